// Host side of the C interface in include/pda.h: argument validation (pure
// host code, no HIP call), the launch plan, the per-(device, stream)
// workspace and the kernel launches of a decode step, a KV append and a
// prefill.

#include "pda.h"
#include "pda_internal.h"

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <initializer_list>
#include <map>
#include <memory>
#include <mutex>
#include <numeric>
#include <string>
#include <tuple>
#include <utility>
#include <vector>

static_assert(pda::kScratchBytes == PDA_NOALLOC_SCRATCH_BYTES, "fixed scratch size differs from the header's");

namespace {

thread_local std::string g_error;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_error = buf;
  return code;
}

int fail_hip(hipError_t e, const char* what) {
  return fail(PDA_EHIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kDefaultWavesPerCu = 8;   // upper bound used by pda_query_plan
constexpr int kDefaultMinShare = 8;     // blocks: below this a wave's fixed costs dominate
// Static split by default: with chunk switches that drain a wave's load
// pipeline, handing out chunks dynamically measured slower on every step
// shape tried (the last chunk's tail outweighs the balance it buys).
constexpr int kDefaultChunksPerWave = 1;
constexpr int64_t kChunkMinBytes = 512 << 10;  // of K and V: a chunk outlasts its start-up costs
constexpr int64_t kAlign = 256;

int64_t align_up(int64_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct PtrAlign {
  const void* p;
  uintptr_t align;
  const char* name;
};

// Null pointers pass (the callers check which ones are required).
int check_alignment(std::initializer_list<PtrAlign> ptrs) {
  for (const PtrAlign& x : ptrs)
    if (reinterpret_cast<uintptr_t>(x.p) % x.align)
      return fail(PDA_EINVAL, "%s is not %d-byte aligned", x.name, (int)x.align);
  return PDA_OK;
}

struct Plan {
  int requested;  // the pda_variant the options asked for
  int Q;          // query tokens per sequence
  pda::Variant variant;
  pda::KvType kv;
  int G;
  int len_cap;
  int waves_per_cu;  // 0 = decide from occupancy at launch
  int min_share;
  int chunks_per_wave;
  int chunk_min;
};

// Validate everything that does not need a device. Returns PDA_OK or an error.
int validate(const pda_problem* pr, const pda_options* op, float softmax_scale, Plan* plan) {
  if (!pr) return fail(PDA_EINVAL, "problem is NULL");
  if (pr->num_seqs < 0) return fail(PDA_EINVAL, "num_seqs = %d < 0", pr->num_seqs);
  if (pr->num_q_heads < 1 || pr->num_kv_heads < 1)
    return fail(PDA_EINVAL, "num_q_heads = %d and num_kv_heads = %d must be >= 1", pr->num_q_heads,
                pr->num_kv_heads);
  if (pr->num_q_heads % pr->num_kv_heads)
    return fail(PDA_EINVAL, "num_q_heads = %d is not a multiple of num_kv_heads = %d", pr->num_q_heads,
                pr->num_kv_heads);
  const int G = pr->num_q_heads / pr->num_kv_heads;
  if (G > pda::kMaxGroup)
    return fail(PDA_EUNSUPPORTED, "GQA group of %d query heads per KV head (max %d)", G, pda::kMaxGroup);
  if (pr->head_dim != 64 && pr->head_dim != 128)
    return fail(PDA_EUNSUPPORTED, "head_dim = %d (supported: 64, 128)", pr->head_dim);
  if (pr->block_size != pda::kBlockSize)
    return fail(PDA_EUNSUPPORTED, "block_size = %d (supported: 16)", pr->block_size);
  if (pr->max_blocks_per_seq < 1) return fail(PDA_EINVAL, "max_blocks_per_seq = %d < 1", pr->max_blocks_per_seq);
  if (pr->num_blocks < 1) return fail(PDA_EINVAL, "num_blocks = %lld < 1", (long long)pr->num_blocks);
  const int64_t table_tokens = (int64_t)pr->max_blocks_per_seq * pda::kBlockSize;
  if (table_tokens > INT32_MAX) return fail(PDA_EINVAL, "max_blocks_per_seq * 16 overflows int32");
  if ((int64_t)pr->num_seqs * ((int64_t)pr->max_blocks_per_seq + pda::kUnitCostPlain) * pr->num_kv_heads > INT32_MAX)
    return fail(PDA_EINVAL, "num_seqs * (max_blocks_per_seq + %d) * num_kv_heads overflows int32", pda::kUnitCostPlain);
  if ((int64_t)pr->num_seqs * pr->num_q_heads > INT32_MAX) return fail(PDA_EINVAL, "num_seqs * num_q_heads too large");
  if (pr->max_seq_len < 0) return fail(PDA_EINVAL, "max_seq_len = %d < 0", pr->max_seq_len);
  if (pr->max_seq_len > table_tokens)
    return fail(PDA_EINVAL, "max_seq_len = %d exceeds max_blocks_per_seq * 16 = %lld", pr->max_seq_len,
                (long long)table_tokens);
  // every cache byte offset must fit int64 (and the tile index p * Hkv + kvh)
  const int64_t tile = (int64_t)pda::kBlockSize * pr->head_dim * 4;
  if (pr->num_blocks > INT64_MAX / pr->num_kv_heads / tile) return fail(PDA_EINVAL, "num_blocks too large");

  const int qd = pr->q_dtype, kd = pr->kv_dtype;
  if (qd != PDA_DTYPE_F32 && qd != PDA_DTYPE_BF16)
    return fail(qd == PDA_DTYPE_FP8_E4M3 ? PDA_EUNSUPPORTED : PDA_EINVAL, "q_dtype = %d (supported: F32, BF16)", qd);
  if (kd != PDA_DTYPE_F32 && kd != PDA_DTYPE_BF16 && kd != PDA_DTYPE_FP8_E4M3)
    return fail(PDA_EINVAL, "kv_dtype = %d is not a pda_dtype", kd);
  if (kd == PDA_DTYPE_F32 && qd != PDA_DTYPE_F32)
    return fail(PDA_EUNSUPPORTED, "an f32 KV cache needs f32 q");
  if (kd != PDA_DTYPE_F32 && qd != PDA_DTYPE_BF16)
    return fail(PDA_EUNSUPPORTED, "a bf16 or fp8 KV cache needs bf16 q");
  if (pr->out_dtype != qd && pr->out_dtype != PDA_DTYPE_F32)
    return fail(PDA_EINVAL, "out_dtype = %d (must be q_dtype or F32)", pr->out_dtype);
  if (!std::isfinite(softmax_scale)) return fail(PDA_EINVAL, "softmax_scale is not finite");
  if (pr->q_tokens < 0) return fail(PDA_EINVAL, "q_tokens = %d < 0", pr->q_tokens);
  const int Q = pr->q_tokens > 1 ? pr->q_tokens : 1;
  if ((int64_t)pr->num_seqs * Q * pr->num_q_heads > INT32_MAX)
    return fail(PDA_EINVAL, "num_seqs * q_tokens * num_q_heads too large");

  int variant = op ? op->variant : PDA_VARIANT_AUTO;
  if (variant != PDA_VARIANT_AUTO && variant != PDA_VARIANT_VECTOR && variant != PDA_VARIANT_MFMA)
    return fail(PDA_EINVAL, "options.variant = %d is not a pda_variant", variant);
  if (Q > 1) {  // several query tokens: MFMA columns are (token, head) pairs
    if (kd == PDA_DTYPE_F32 || variant == PDA_VARIANT_VECTOR)
      return fail(PDA_EUNSUPPORTED, "q_tokens > 1 runs on the MFMA kernel: it needs a bf16 or fp8 KV cache");
    if (Q * G > pda::kWideColumns)
      return fail(PDA_EUNSUPPORTED, "q_tokens * (num_q_heads / num_kv_heads) = %d exceeds %d", Q * G,
                  pda::kWideColumns);
    variant = PDA_VARIANT_MFMA;
  }
  if (variant == PDA_VARIANT_AUTO)
    variant = (kd != PDA_DTYPE_F32 && G >= 4) ? PDA_VARIANT_MFMA : PDA_VARIANT_VECTOR;
  if (variant == PDA_VARIANT_MFMA && kd == PDA_DTYPE_F32)
    return fail(PDA_EUNSUPPORTED, "the MFMA kernel needs a bf16 or fp8 KV cache");
  if (variant == PDA_VARIANT_VECTOR && G > pda::kMaxGroupVector)
    return fail(PDA_EUNSUPPORTED, "the vector kernel handles at most %d query heads per KV head (got %d)",
                pda::kMaxGroupVector, G);
  if (op && (op->waves_per_cu < 0 || op->waves_per_cu > 64))
    return fail(PDA_EINVAL, "options.waves_per_cu = %d (0..64)", op->waves_per_cu);
  if (op && op->min_blocks_per_wave < 0)
    return fail(PDA_EINVAL, "options.min_blocks_per_wave = %d < 0", op->min_blocks_per_wave);
  if (op && (op->chunks_per_wave < 0 || op->chunks_per_wave > 64))
    return fail(PDA_EINVAL, "options.chunks_per_wave = %d (0..64)", op->chunks_per_wave);
  if (op && op->min_blocks_per_chunk < 0)
    return fail(PDA_EINVAL, "options.min_blocks_per_chunk = %d < 0", op->min_blocks_per_chunk);

  plan->requested = op ? op->variant : PDA_VARIANT_AUTO;
  plan->variant = variant == PDA_VARIANT_MFMA ? pda::Variant::Mfma : pda::Variant::Vector;
  plan->kv = kd == PDA_DTYPE_F32 ? pda::KvType::F32 : (kd == PDA_DTYPE_BF16 ? pda::KvType::BF16 : pda::KvType::FP8);
  plan->G = G;
  plan->Q = Q;
  plan->len_cap = pr->max_seq_len > 0 ? pr->max_seq_len : (int)table_tokens;
  plan->waves_per_cu = op ? op->waves_per_cu : 0;
  plan->min_share = (op && op->min_blocks_per_wave > 0) ? op->min_blocks_per_wave : kDefaultMinShare;
  plan->chunks_per_wave = (op && op->chunks_per_wave > 0) ? op->chunks_per_wave : kDefaultChunksPerWave;
  const int esz = kd == PDA_DTYPE_F32 ? 4 : (kd == PDA_DTYPE_BF16 ? 2 : 1);
  const int64_t block_head_bytes = 2LL * pda::kBlockSize * pr->head_dim * esz;
  plan->chunk_min = (op && op->min_blocks_per_chunk > 0) ? op->min_blocks_per_chunk
                                                         : (int)(kChunkMinBytes / block_head_bytes);
  return PDA_OK;
}

// Shared-prefix mode: groups of group_size consecutive sequences; each
// group's shared blocks become nsub work entries of M members (M * G <= 32
// query columns), ahead of one entry per sequence for the rest of it.
struct Groups {
  bool on = false;
  int group_size = 1, M = 1, nsub = 0, num_groups = 0;
  int64_t n_prefix = 0;
  const int32_t* shared_blocks = nullptr;
};

int validate_groups(const pda_problem* pr, int32_t group_size, const int32_t* shared_blocks, Plan* plan,
                    Groups* gr) {
  if (group_size < 1) return fail(PDA_EINVAL, "group_size = %d < 1", group_size);
  if (pr->num_seqs % group_size)
    return fail(PDA_EINVAL, "num_seqs = %d is not a multiple of group_size = %d", pr->num_seqs, group_size);
  if (plan->kv == pda::KvType::F32)
    return fail(PDA_EUNSUPPORTED, "shared-prefix decode runs on the MFMA kernel: it needs a bf16 or fp8 KV cache");
  if (plan->requested == PDA_VARIANT_VECTOR)
    return fail(PDA_EUNSUPPORTED, "shared-prefix decode runs on the MFMA kernel, not the vector kernel");
  if (pr->num_seqs > 0 && !shared_blocks) return fail(PDA_EINVAL, "shared_blocks is NULL");
  if (plan->Q > 1) return fail(PDA_EUNSUPPORTED, "shared-prefix decode takes one query token per sequence");
  plan->variant = pda::Variant::Mfma;
  gr->on = true;
  gr->group_size = group_size;
  const int per = pda::kWideColumns / plan->G;  // members whose heads fill two MFMA N-tiles
  gr->M = group_size < per ? group_size : (per > 0 ? per : 1);
  gr->nsub = (group_size + gr->M - 1) / gr->M;
  gr->num_groups = pr->num_seqs / group_size;
  gr->n_prefix = (int64_t)gr->num_groups * gr->nsub;
  gr->shared_blocks = shared_blocks;
  if ((gr->n_prefix + pr->num_seqs) * pr->num_kv_heads *
          ((int64_t)pr->max_blocks_per_seq + pda::kUnitCostShared) > INT32_MAX)
    return fail(PDA_EINVAL, "(entries) * num_kv_heads * (max_blocks_per_seq + %d) overflows int32",
                pda::kUnitCostShared);
  return PDA_OK;
}

struct Layout {
  int64_t hdr, sg, cum, m, l, acc, total;
};

// header | sg[num_groups] | cum[entries] | m, l [slots, Gp] | acc [slots, Gp, D]
Layout workspace_layout(const pda_problem* pr, const Plan& plan, const Groups& gr, int chunks_max) {
  Layout w;
  const int64_t entries = gr.n_prefix + pr->num_seqs;
  const int64_t gp = gr.on ? (int64_t)gr.M * plan.G : (int64_t)plan.Q * plan.G;
  const int64_t slots = pda::partial_slots(entries, pr->num_kv_heads, chunks_max);
  w.hdr = 0;
  w.sg = align_up(pda::kHdrWords * 4);
  w.cum = w.sg + align_up((int64_t)gr.num_groups * 4);
  w.m = w.cum + align_up(entries * 4);
  w.l = w.m + align_up(slots * gp * 4);
  w.acc = w.l + align_up(slots * gp * 4);
  w.total = w.acc + align_up(slots * gp * pr->head_dim * 4);
  return w;
}

// ------------------------------------------------------------- device state

struct DeviceInfo {
  bool ok = false;
  int cus = 0;
  std::string arch;
};

struct Workspace {
  std::mutex mu;
  void* ptr = nullptr;
  int64_t bytes = 0;
  // The combine kernel zeroes the chunk counter after each decode kernel; if a
  // combine launch failed, the next call zeroes it first.
  bool rearm = false;
  // A graph captured on the stream holds `ptr`: growth then keeps the old
  // allocation (in `retired`) so that replays stay valid.
  bool captured = false;
  std::vector<void*> retired;
};

// The no-allocation entry point's per-device state: the device address of
// that device's copy of the fixed scratch array (looked up on the first call
// with the device current) and the counter re-arm flag. A fixed table, so
// that the entry point allocates nothing, not even host memory for its state.
constexpr int kMaxDevices = 64;
struct FixedScratch {
  std::mutex mu;
  void* ptr = nullptr;
  bool rearm = false;
};
FixedScratch g_fixed[kMaxDevices];

std::mutex g_mu;
std::map<int, DeviceInfo> g_devices;
std::map<std::pair<int, hipStream_t>, std::unique_ptr<Workspace>> g_workspaces;
std::map<std::tuple<int, int, int, int, int>, int> g_occupancy;

int device_info(int dev, DeviceInfo* out) {
  std::lock_guard<std::mutex> lk(g_mu);
  auto it = g_devices.find(dev);
  if (it != g_devices.end()) {
    *out = it->second;
    return PDA_OK;
  }
  DeviceInfo d;
  hipDeviceProp_t prop;
  hipError_t e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDeviceProperties");
  d.cus = prop.multiProcessorCount;
  d.arch = prop.gcnArchName;
  d.ok = d.arch.rfind("gfx950", 0) == 0;
  g_devices[dev] = d;
  *out = d;
  return PDA_OK;
}

int occupancy(int dev, pda::Variant v, pda::KvType kv, int D, int G, bool wide, int* wgs) {
  const int gb = v == pda::Variant::Mfma ? (wide ? pda::kWideColumns : 16) : (G <= 1 ? 1 : G <= 2 ? 2 : G <= 4 ? 4 : 8);
  auto key = std::make_tuple(dev, (int)v, (int)kv, D, gb);
  {
    std::lock_guard<std::mutex> lk(g_mu);
    auto it = g_occupancy.find(key);
    if (it != g_occupancy.end()) {
      *wgs = it->second;
      return PDA_OK;
    }
  }
  int n = 0;
  hipError_t e = pda::decode_occupancy(v, kv, D, G, wide, &n);
  if (e != hipSuccess) return fail_hip(e, "hipOccupancyMaxActiveBlocksPerMultiprocessor");
  if (n < 1) n = 1;
  std::lock_guard<std::mutex> lk(g_mu);
  g_occupancy[key] = n;
  *wgs = n;
  return PDA_OK;
}

Workspace* workspace_for(int dev, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_mu);
  auto& slot = g_workspaces[std::make_pair(dev, s)];
  if (!slot) slot.reset(new Workspace);
  return slot.get();
}

// True while `s` records into a HIP graph: allocation, frees, waits and
// memsets must then stay out of the call.
bool capturing(hipStream_t s) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  return hipStreamIsCapturing(s, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone;
}

// Grow ws (caller holds ws->mu) to at least `bytes`; growth waits for `s`.
int ensure_workspace(Workspace* ws, int64_t bytes, hipStream_t s) {
  const bool cap = capturing(s);
  if (cap) ws->captured = true;
  if (ws->bytes >= bytes) return PDA_OK;
  if (cap)
    return fail(PDA_EINVAL,
                "the stream's workspace must grow to %lld bytes, which cannot be recorded into a graph: make one "
                "call of this size (or larger) on the stream before capturing it",
                (long long)bytes);
  hipError_t e;
  if (ws->ptr) {
    if (ws->captured) {
      ws->retired.push_back(ws->ptr);
    } else {
      if ((e = hipStreamSynchronize(s)) != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
      if ((e = hipFree(ws->ptr)) != hipSuccess) return fail_hip(e, "hipFree");
    }
    ws->ptr = nullptr;
    ws->bytes = 0;
  }
  const int64_t want = bytes + bytes / 4;  // headroom so small growth does not reallocate
  if ((e = hipMalloc(&ws->ptr, (size_t)want)) != hipSuccess) {
    ws->ptr = nullptr;
    return fail(PDA_ENOMEM, "hipMalloc(%lld) of the workspace: %s", (long long)want, hipGetErrorString(e));
  }
  ws->bytes = want;
  ws->rearm = false;
  if ((e = hipMemsetAsync(ws->ptr, 0, pda::kHdrWords * 4, s)) != hipSuccess) return fail_hip(e, "hipMemsetAsync");
  return PDA_OK;
}

}  // namespace

extern "C" {

int pda_version(void) { return PDA_VERSION; }

const char* pda_last_error(void) { return g_error.c_str(); }

}  // extern "C"

namespace {

int query_plan(const pda_problem* problem, const pda_options* options, float softmax_scale,
               int32_t num_compute_units, const int32_t* group_size, pda_plan_info* info) {
  g_error.clear();
  if (!info) return fail(PDA_EINVAL, "info is NULL");
  if (num_compute_units < 1) return fail(PDA_EINVAL, "num_compute_units = %d < 1", num_compute_units);
  Plan plan;
  int rc = validate(problem, options, softmax_scale, &plan);
  if (rc != PDA_OK) return rc;
  Groups gr;
  static const int32_t kAny = 0;  // shared_blocks is not read by a plan query
  if (group_size && (rc = validate_groups(problem, *group_size, &kAny, &plan, &gr)) != PDA_OK) return rc;
  const int wpc = plan.waves_per_cu > 0 ? plan.waves_per_cu : kDefaultWavesPerCu;
  if ((int64_t)num_compute_units * wpc * plan.chunks_per_wave > INT32_MAX)
    return fail(PDA_EINVAL, "num_compute_units = %d is too large", num_compute_units);
  info->variant = plan.variant == pda::Variant::Mfma ? PDA_VARIANT_MFMA : PDA_VARIANT_VECTOR;
  info->waves = num_compute_units * wpc;
  info->group_size = plan.G;
  info->chunks_max = info->waves * plan.chunks_per_wave;
  info->workspace_bytes = workspace_layout(problem, plan, gr, info->chunks_max).total;
  return PDA_OK;
}

// fixed_scratch: take the workspace from the device's fixed scratch array
// (pda_paged_decode_attention_noalloc) instead of the stream's allocation.
int run(const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table,
        const int32_t* seq_lens, const float* kv_scales, void* out, float softmax_scale,
        const int32_t* group_size, const int32_t* shared_blocks, const pda_problem* problem,
        const pda_options* options, hipStream_t stream, bool fixed_scratch = false) {
  g_error.clear();
  Plan plan;
  int rc = validate(problem, options, softmax_scale, &plan);
  if (rc != PDA_OK) return rc;
  Groups gr;
  if (group_size && (rc = validate_groups(problem, *group_size, shared_blocks, &plan, &gr)) != PDA_OK) return rc;
  if (problem->num_seqs == 0) return PDA_OK;
  if (!q || !k_cache || !v_cache || !block_table || !seq_lens || !out)
    return fail(PDA_EINVAL, "a required pointer (q, k_cache, v_cache, block_table, seq_lens, out) is NULL");
  if (problem->kv_dtype == PDA_DTYPE_FP8_E4M3 && !kv_scales)
    return fail(PDA_EINVAL, "an fp8 KV cache needs kv_scales");
  if ((rc = check_alignment({{q, 16, "q"}, {k_cache, 16, "k_cache"}, {v_cache, 16, "v_cache"}, {out, 16, "out"},
                             {block_table, 4, "block_table"}, {seq_lens, 4, "seq_lens"},
                             {kv_scales, 4, "kv_scales"}})) != PDA_OK)
    return rc;

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  DeviceInfo di;
  if ((rc = device_info(dev, &di)) != PDA_OK) return rc;
  if (!di.ok) return fail(PDA_EUNSUPPORTED, "device %d is %s; this library is built for gfx950", dev, di.arch.c_str());

  int wpc = plan.waves_per_cu;
  if (wpc == 0) {
    const bool wide = (gr.on ? gr.M * plan.G : plan.Q * plan.G) > 16;
    if ((rc = occupancy(dev, plan.variant, plan.kv, problem->head_dim, plan.G, wide, &wpc)) != PDA_OK) return rc;
    if (wpc > kDefaultWavesPerCu) wpc = kDefaultWavesPerCu;
  }
  const int waves = di.cus * wpc;
  const int chunks_max = waves * plan.chunks_per_wave;
  const Layout lay = workspace_layout(problem, plan, gr, chunks_max);

  std::unique_lock<std::mutex> lk;
  char* base = nullptr;
  bool* rearm = nullptr;
  if (fixed_scratch) {
    if (dev < 0 || dev >= kMaxDevices) return fail(PDA_EUNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
    if (lay.total > pda::kScratchBytes)
      return fail(PDA_EINVAL,
                  "this call needs %lld bytes of workspace; the no-allocation entry point's fixed scratch holds %lld "
                  "(fewer sequences, KV heads or waves per call, or pda_paged_decode_attention)",
                  (long long)lay.total, (long long)pda::kScratchBytes);
    FixedScratch* fs = &g_fixed[dev];
    lk = std::unique_lock<std::mutex>(fs->mu);
    if (!fs->ptr) {  // first call on this device (current here): its copy of the array
      void* p = nullptr;
      if ((e = pda::scratch_address(&p)) != hipSuccess) return fail_hip(e, "hipGetSymbolAddress(scratch)");
      fs->ptr = p;
    }
    base = static_cast<char*>(fs->ptr);
    rearm = &fs->rearm;
  } else {
    Workspace* ws = workspace_for(dev, stream);
    lk = std::unique_lock<std::mutex>(ws->mu);
    if ((rc = ensure_workspace(ws, lay.total, stream)) != PDA_OK) return rc;
    base = static_cast<char*>(ws->ptr);
    rearm = &ws->rearm;
  }
  if (*rearm) {
    if (capturing(stream))
      return fail(PDA_EINVAL, "the workspace needs a reset after a failed launch: make one call outside capture");
    if ((e = hipMemsetAsync(base + pda::kHdrNext * 4, 0, 4, stream)) != hipSuccess)
      return fail_hip(e, "hipMemsetAsync");
    *rearm = false;
  }

  pda::DecodeArgs a;
  a.q = q;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.kv_scales = kv_scales;
  a.out = out;
  a.scale_log2 = softmax_scale * 1.4426950408889634f;
  a.mfma_scale_log2 = std::fabs(softmax_scale) * 1.4426950408889634f;
  a.neg_scale = softmax_scale < 0.f;
  a.B = problem->num_seqs;
  a.Hq = problem->num_q_heads;
  a.Hkv = problem->num_kv_heads;
  a.G = plan.G;
  a.D = problem->head_dim;
  a.max_blocks = problem->max_blocks_per_seq;
  a.num_blocks = problem->num_blocks;
  a.len_cap = plan.len_cap;
  a.min_share = plan.min_share;
  a.chunk_min = plan.chunk_min;
  a.chunks_max = chunks_max;
  a.waves = waves;
  // Workgroups of 4 (or 2) independent waves when every CU gets whole groups:
  // fewer, larger workgroups dispatch faster than one-wave groups.
  a.waves_per_group = wpc % 4 == 0 ? 4 : (wpc % 2 == 0 ? 2 : 1);
  a.out_bf16 = problem->out_dtype == PDA_DTYPE_BF16;
  a.E = (int32_t)(gr.n_prefix + problem->num_seqs);
  a.shared = gr.on ? 1 : 0;
  a.group_size = gr.group_size;
  a.M = gr.M;
  a.nsub = gr.nsub;
  a.n_prefix = (int32_t)gr.n_prefix;
  a.Gp = gr.on ? gr.M * plan.G : plan.Q * plan.G;
  a.Qn = plan.Q;
  a.shared_blocks = gr.shared_blocks;
  a.sg = reinterpret_cast<int32_t*>(base + lay.sg);
  a.hdr = reinterpret_cast<int32_t*>(base + lay.hdr);
  a.share = a.hdr + pda::kHdrShare;
  a.cum = reinterpret_cast<int32_t*>(base + lay.cum);
  a.ws_m = reinterpret_cast<float*>(base + lay.m);
  a.ws_l = reinterpret_cast<float*>(base + lay.l);
  a.ws_acc = reinterpret_cast<float*>(base + lay.acc);
  if (gr.on && (e = pda::launch_prefix(a, gr.num_groups, stream)) != hipSuccess)
    return fail_hip(e, "prefix kernel launch");
  if ((e = pda::launch_decode(a, plan.variant, plan.kv, stream)) != hipSuccess)
    return fail_hip(e, "decode kernel launch");
  if ((e = pda::launch_combine(a, stream)) != hipSuccess) {
    *rearm = true;
    return fail_hip(e, "combine kernel launch");
  }
  return PDA_OK;
}

int append_run(const void* k_new, const void* v_new, void* k_cache, void* v_cache, float* kv_scales,
               const int32_t* block_table, const int32_t* positions, const pda_append_problem* pr,
               hipStream_t stream) {
  g_error.clear();
  if (!pr) return fail(PDA_EINVAL, "problem is NULL");
  if (pr->num_seqs < 0) return fail(PDA_EINVAL, "num_seqs = %d < 0", pr->num_seqs);
  if (pr->num_kv_heads < 1) return fail(PDA_EINVAL, "num_kv_heads = %d < 1", pr->num_kv_heads);
  if (pr->head_dim != 64 && pr->head_dim != 128)
    return fail(PDA_EUNSUPPORTED, "head_dim = %d (supported: 64, 128)", pr->head_dim);
  if (pr->block_size != pda::kBlockSize)
    return fail(PDA_EUNSUPPORTED, "block_size = %d (supported: 16)", pr->block_size);
  if (pr->max_blocks_per_seq < 1) return fail(PDA_EINVAL, "max_blocks_per_seq = %d < 1", pr->max_blocks_per_seq);
  if ((int64_t)pr->max_blocks_per_seq * pda::kBlockSize > INT32_MAX)
    return fail(PDA_EINVAL, "max_blocks_per_seq * 16 overflows int32");
  if ((int64_t)pr->num_seqs * pr->num_kv_heads > INT32_MAX) return fail(PDA_EINVAL, "num_seqs * num_kv_heads too large");
  if (pr->num_blocks < 1) return fail(PDA_EINVAL, "num_blocks = %lld < 1", (long long)pr->num_blocks);
  const int64_t tile = (int64_t)pda::kBlockSize * pr->head_dim * 4;
  if (pr->num_blocks > INT64_MAX / pr->num_kv_heads / tile) return fail(PDA_EINVAL, "num_blocks too large");
  if (pr->new_dtype != PDA_DTYPE_F32 && pr->new_dtype != PDA_DTYPE_BF16)
    return fail(PDA_EINVAL, "new_dtype = %d (supported: F32, BF16)", pr->new_dtype);
  const int kd = pr->kv_dtype;
  if (kd != PDA_DTYPE_F32 && kd != PDA_DTYPE_BF16 && kd != PDA_DTYPE_FP8_E4M3)
    return fail(PDA_EINVAL, "kv_dtype = %d is not a pda_dtype", kd);
  if (pr->num_seqs == 0) return PDA_OK;
  if (!k_new || !v_new || !k_cache || !v_cache || !block_table || !positions)
    return fail(PDA_EINVAL, "a required pointer (k_new, v_new, k_cache, v_cache, block_table, positions) is NULL");
  if (kd == PDA_DTYPE_FP8_E4M3 && !kv_scales) return fail(PDA_EINVAL, "an fp8 KV cache needs kv_scales");

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  DeviceInfo di;
  int rc;
  if ((rc = device_info(dev, &di)) != PDA_OK) return rc;
  if (!di.ok) return fail(PDA_EUNSUPPORTED, "device %d is %s; this library is built for gfx950", dev, di.arch.c_str());
  Workspace* ws = workspace_for(dev, stream);
  std::lock_guard<std::mutex> lk(ws->mu);
  if ((rc = ensure_workspace(ws, align_up(pda::kHdrWords * 4), stream)) != PDA_OK) return rc;

  pda::AppendArgs a;
  a.k_new = k_new;
  a.v_new = v_new;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.kv_scales = kv_scales;
  a.block_table = block_table;
  a.positions = positions;
  a.B = pr->num_seqs;
  a.Hkv = pr->num_kv_heads;
  a.D = pr->head_dim;
  a.max_blocks = pr->max_blocks_per_seq;
  a.num_blocks = pr->num_blocks;
  a.new_bf16 = pr->new_dtype == PDA_DTYPE_BF16;
  a.status = static_cast<int32_t*>(ws->ptr) + pda::kHdrStatus;
  const pda::KvType kv = kd == PDA_DTYPE_F32 ? pda::KvType::F32
                         : kd == PDA_DTYPE_BF16 ? pda::KvType::BF16 : pda::KvType::FP8;
  if ((e = pda::launch_append(a, kv, stream)) != hipSuccess) return fail_hip(e, "append kernel launch");
  return PDA_OK;
}

// Largest prefill image in bytes: PDA_PREFILL_IMAGE_MAX_MB (MiB, read on each
// call; 0 always stages through registers), 8 GiB by default.
int64_t prefill_image_cap() {
  const char* v = std::getenv("PDA_PREFILL_IMAGE_MAX_MB");
  if (!v || !*v) return 8ll << 30;
  char* end = nullptr;
  const long long mb = std::strtoll(v, &end, 10);
  if (end == v || mb < 0) return 8ll << 30;
  return mb > (INT64_MAX >> 20) ? INT64_MAX : (int64_t)mb << 20;
}

int prefill_run(const void* q, const int32_t* q_offsets, const void* k_cache, const void* v_cache,
                const int32_t* block_table, const int32_t* seq_lens, const float* kv_scales, void* out,
                float softmax_scale, const pda_prefill_problem* pr, hipStream_t stream) {
  g_error.clear();
  if (!pr) return fail(PDA_EINVAL, "problem is NULL");
  if (pr->num_seqs < 0) return fail(PDA_EINVAL, "num_seqs = %d < 0", pr->num_seqs);
  if (pr->num_tokens < 0) return fail(PDA_EINVAL, "num_tokens = %d < 0", pr->num_tokens);
  if (pr->num_q_heads < 1 || pr->num_kv_heads < 1)
    return fail(PDA_EINVAL, "num_q_heads = %d and num_kv_heads = %d must be >= 1", pr->num_q_heads,
                pr->num_kv_heads);
  if (pr->num_q_heads % pr->num_kv_heads)
    return fail(PDA_EINVAL, "num_q_heads = %d is not a multiple of num_kv_heads = %d", pr->num_q_heads,
                pr->num_kv_heads);
  const int G = pr->num_q_heads / pr->num_kv_heads;
  if (G > pda::kMaxGroup)
    return fail(PDA_EUNSUPPORTED, "GQA group of %d query heads per KV head (max %d)", G, pda::kMaxGroup);
  if (pr->head_dim != 64 && pr->head_dim != 128)
    return fail(PDA_EUNSUPPORTED, "head_dim = %d (supported: 64, 128)", pr->head_dim);
  if (pr->block_size != pda::kBlockSize)
    return fail(PDA_EUNSUPPORTED, "block_size = %d (supported: 16)", pr->block_size);
  if (pr->max_blocks_per_seq < 1) return fail(PDA_EINVAL, "max_blocks_per_seq = %d < 1", pr->max_blocks_per_seq);
  if (pr->num_blocks < 1) return fail(PDA_EINVAL, "num_blocks = %lld < 1", (long long)pr->num_blocks);
  const int64_t table_tokens = (int64_t)pr->max_blocks_per_seq * pda::kBlockSize;
  if (table_tokens > INT32_MAX) return fail(PDA_EINVAL, "max_blocks_per_seq * 16 overflows int32");
  if ((int64_t)pr->num_seqs * pr->max_blocks_per_seq > INT32_MAX)
    return fail(PDA_EINVAL, "num_seqs * max_blocks_per_seq overflows int32");
  if ((int64_t)pr->num_tokens * pr->num_q_heads > INT32_MAX)
    return fail(PDA_EINVAL, "num_tokens * num_q_heads overflows int32");
  if (pr->max_seq_len < 0) return fail(PDA_EINVAL, "max_seq_len = %d < 0", pr->max_seq_len);
  if (pr->max_seq_len > table_tokens)
    return fail(PDA_EINVAL, "max_seq_len = %d exceeds max_blocks_per_seq * 16 = %lld", pr->max_seq_len,
                (long long)table_tokens);
  const int64_t tile = (int64_t)pda::kBlockSize * pr->head_dim * 4;
  if (pr->num_blocks > INT64_MAX / pr->num_kv_heads / tile) return fail(PDA_EINVAL, "num_blocks too large");
  if (pr->q_dtype != PDA_DTYPE_BF16)
    return fail(pr->q_dtype == PDA_DTYPE_F32 ? PDA_EUNSUPPORTED : PDA_EINVAL, "q_dtype = %d (supported: BF16)",
                pr->q_dtype);
  const int kd = pr->kv_dtype;
  if (kd == PDA_DTYPE_F32) return fail(PDA_EUNSUPPORTED, "prefill runs on the matrix cores: it needs a bf16 or fp8 cache");
  if (kd != PDA_DTYPE_BF16 && kd != PDA_DTYPE_FP8_E4M3) return fail(PDA_EINVAL, "kv_dtype = %d is not a pda_dtype", kd);
  if (pr->out_dtype != PDA_DTYPE_BF16 && pr->out_dtype != PDA_DTYPE_F32)
    return fail(PDA_EINVAL, "out_dtype = %d (must be BF16 or F32)", pr->out_dtype);
  if (!std::isfinite(softmax_scale)) return fail(PDA_EINVAL, "softmax_scale is not finite");
  const int TQ = pda::kPfColumns / G;
  // every sequence's tiles: sum of ceil(n_b / TQ) <= (T + B (TQ - 1)) / TQ
  const int64_t items_max = ((int64_t)pr->num_tokens + (int64_t)pr->num_seqs * (TQ - 1)) / TQ;
  // the attention grid names a claimed unit (item, KV head) as 8 * index + queue in an int32
  if (items_max * pr->num_kv_heads > INT32_MAX / 8)
    return fail(PDA_EINVAL, "too many work units (%lld tiles x %d KV heads) for the unit queues", (long long)items_max,
                pr->num_kv_heads);
  if (pr->num_seqs == 0 || pr->num_tokens == 0) return PDA_OK;
  if (!q || !q_offsets || !k_cache || !v_cache || !block_table || !seq_lens || !out)
    return fail(PDA_EINVAL, "a required pointer (q, q_offsets, k_cache, v_cache, block_table, seq_lens, out) is NULL");
  if (kd == PDA_DTYPE_FP8_E4M3 && !kv_scales) return fail(PDA_EINVAL, "an fp8 KV cache needs kv_scales");
  {
    const int rc = check_alignment({{q, 16, "q"}, {k_cache, 16, "k_cache"}, {v_cache, 16, "v_cache"},
                                    {out, 16, "out"}, {q_offsets, 4, "q_offsets"}, {block_table, 4, "block_table"},
                                    {seq_lens, 4, "seq_lens"}, {kv_scales, 4, "kv_scales"}});
    if (rc != PDA_OK) return rc;
  }

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  DeviceInfo di;
  int rc;
  if ((rc = device_info(dev, &di)) != PDA_OK) return rc;
  if (!di.ok) return fail(PDA_EUNSUPPORTED, "device %d is %s; this library is built for gfx950", dev, di.arch.c_str());
  Workspace* ws = workspace_for(dev, stream);
  std::lock_guard<std::mutex> lk(ws->mu);
  const int64_t items_off = align_up(pda::kHdrWords * 4);
  const int64_t plain_bytes = items_off + items_max * 16;
  // The image (V in fp16; for an fp8 cache K in bf16 too) follows the work
  // list when it fits the cap; a capture that cannot grow the workspace, or a
  // failed allocation, takes the staging kernel, whose results are the same.
  const int64_t img_half = pr->num_blocks * pr->num_kv_heads * (int64_t)pda::kBlockSize * pr->head_dim * 2;
  const int64_t img_bytes = kd == PDA_DTYPE_FP8_E4M3 ? 2 * img_half : img_half;
  const int64_t img_off = align_up(plain_bytes);
  bool use_img = img_bytes <= prefill_image_cap();
  if (use_img && capturing(stream) && ws->bytes < img_off + img_bytes) use_img = false;
  if (use_img) {
    rc = ensure_workspace(ws, img_off + img_bytes, stream);
    if (rc == PDA_ENOMEM) {
      use_img = false;
      g_error.clear();
    } else if (rc != PDA_OK) {
      return rc;
    }
  }
  if (!use_img && (rc = ensure_workspace(ws, plain_bytes, stream)) != PDA_OK) return rc;
  char* base = static_cast<char*>(ws->ptr);

  pda::PrefillArgs a;
  a.q = q;
  a.q_offsets = q_offsets;
  a.k_cache = k_cache;
  a.v_cache = v_cache;
  a.block_table = block_table;
  a.seq_lens = seq_lens;
  a.kv_scales = kv_scales;
  a.out = out;
  a.scale_log2 = std::fabs(softmax_scale) * 1.4426950408889634f;
  a.neg_scale = softmax_scale < 0.f;
  a.B = pr->num_seqs;
  a.T = pr->num_tokens;
  a.Hq = pr->num_q_heads;
  a.Hkv = pr->num_kv_heads;
  a.G = G;
  a.D = pr->head_dim;
  a.TQ = TQ;
  a.max_blocks = pr->max_blocks_per_seq;
  a.num_blocks = pr->num_blocks;
  a.len_cap = pr->max_seq_len > 0 ? pr->max_seq_len : (int)table_tokens;
  int shift = 0;
  while ((a.len_cap >> shift) >= pda::kPfBuckets) ++shift;
  a.len_shift = shift;
  a.items_max = (int32_t)items_max;
  a.out_bf16 = pr->out_dtype == PDA_DTYPE_BF16;
  a.cus = di.cus;
  a.nq = std::gcd(a.Hkv, 8);
  a.hdr = reinterpret_cast<int32_t*>(base);
  a.items = reinterpret_cast<int4*>(base + items_off);
  a.v_img = use_img ? base + img_off : nullptr;
  a.k_img = use_img && kd == PDA_DTYPE_FP8_E4M3 ? base + img_off + img_half : nullptr;
  const pda::KvType kv = kd == PDA_DTYPE_BF16 ? pda::KvType::BF16 : pda::KvType::FP8;
  if ((e = pda::launch_prefill(a, kv, stream)) != hipSuccess) return fail_hip(e, "prefill kernel launch");
  return PDA_OK;
}

}  // namespace

extern "C" {

int pda_query_plan(const pda_problem* problem, const pda_options* options, float softmax_scale,
                   int32_t num_compute_units, pda_plan_info* info) {
  return query_plan(problem, options, softmax_scale, num_compute_units, nullptr, info);
}

int pda_query_plan_shared_prefix(const pda_problem* problem, const pda_options* options, float softmax_scale,
                                 int32_t group_size, int32_t num_compute_units, pda_plan_info* info) {
  return query_plan(problem, options, softmax_scale, num_compute_units, &group_size, info);
}

int pda_paged_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                               const int32_t* block_table, const int32_t* seq_lens, const float* kv_scales,
                               void* out, float softmax_scale, const pda_problem* problem,
                               const pda_options* options, hipStream_t stream) {
  return run(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale, nullptr, nullptr,
             problem, options, stream);
}

int pda_paged_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* block_table, const int32_t* seq_lens, const float* kv_scales,
                                       void* out, float softmax_scale, const pda_problem* problem,
                                       const pda_options* options, hipStream_t stream) {
  return run(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale, nullptr, nullptr,
             problem, options, stream, /*fixed_scratch=*/true);
}

int pda_paged_kv_append(const void* k_new, const void* v_new, void* k_cache, void* v_cache, float* kv_scales,
                        const int32_t* block_table, const int32_t* positions, const pda_append_problem* problem,
                        hipStream_t stream) {
  return append_run(k_new, v_new, k_cache, v_cache, kv_scales, block_table, positions, problem, stream);
}

int pda_paged_decode_attention_shared_prefix(const void* q, const void* k_cache, const void* v_cache,
                                             const int32_t* block_table, const int32_t* seq_lens,
                                             const float* kv_scales, void* out, float softmax_scale,
                                             int32_t group_size, const int32_t* shared_blocks,
                                             const pda_problem* problem, const pda_options* options,
                                             hipStream_t stream) {
  return run(q, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale, &group_size,
             shared_blocks, problem, options, stream);
}

int pda_paged_prefill_attention(const void* q, const int32_t* q_offsets, const void* k_cache, const void* v_cache,
                                const int32_t* block_table, const int32_t* seq_lens, const float* kv_scales,
                                void* out, float softmax_scale, const pda_prefill_problem* problem,
                                hipStream_t stream) {
  return prefill_run(q, q_offsets, k_cache, v_cache, block_table, seq_lens, kv_scales, out, softmax_scale, problem,
                     stream);
}

int pda_read_device_status(hipStream_t stream) {
  g_error.clear();
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  Workspace* ws = workspace_for(dev, stream);
  std::lock_guard<std::mutex> lk(ws->mu);
  if ((e = hipStreamSynchronize(stream)) != hipSuccess) return fail_hip(e, "hipStreamSynchronize");
  // the current workspace and any a captured graph still writes to
  int32_t all = 0;
  for (void* p : ws->retired) {
    int32_t word = 0;
    int32_t* hdr = static_cast<int32_t*>(p) + pda::kHdrStatus;
    if ((e = hipMemcpy(&word, hdr, 4, hipMemcpyDeviceToHost)) != hipSuccess) return fail_hip(e, "hipMemcpy");
    if (word && (e = hipMemset(hdr, 0, 4)) != hipSuccess) return fail_hip(e, "hipMemset");
    all |= word;
  }
  if (ws->ptr) {
    int32_t word = 0;
    int32_t* hdr = static_cast<int32_t*>(ws->ptr) + pda::kHdrStatus;
    if ((e = hipMemcpy(&word, hdr, 4, hipMemcpyDeviceToHost)) != hipSuccess) return fail_hip(e, "hipMemcpy");
    if (word && (e = hipMemset(hdr, 0, 4)) != hipSuccess) return fail_hip(e, "hipMemset");
    all |= word;
  }
  // the device's fixed scratch, once the no-allocation entry point has used it
  if (dev >= 0 && dev < kMaxDevices) {
    FixedScratch* fs = &g_fixed[dev];
    std::lock_guard<std::mutex> fl(fs->mu);
    if (fs->ptr) {
      int32_t word = 0;
      int32_t* hdr = static_cast<int32_t*>(fs->ptr) + pda::kHdrStatus;
      if ((e = hipMemcpy(&word, hdr, 4, hipMemcpyDeviceToHost)) != hipSuccess) return fail_hip(e, "hipMemcpy");
      if (word && (e = hipMemset(hdr, 0, 4)) != hipSuccess) return fail_hip(e, "hipMemset");
      all |= word;
    }
  }
  return all;
}

int pda_release_workspaces(void) {
  g_error.clear();
  std::lock_guard<std::mutex> lk(g_mu);
  int rc = PDA_OK;
  int cur = 0;
  const bool have_dev = hipGetDevice(&cur) == hipSuccess;
  for (auto& kv : g_workspaces) {
    Workspace* ws = kv.second.get();
    std::lock_guard<std::mutex> wl(ws->mu);
    if (!ws->ptr && ws->retired.empty()) continue;
    hipError_t e = hipSetDevice(kv.first.first);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e == hipSuccess && ws->ptr) e = hipFree(ws->ptr);
    for (void* p : ws->retired)
      if (e == hipSuccess) e = hipFree(p);
    if (e != hipSuccess) rc = fail_hip(e, "releasing a workspace");
    ws->ptr = nullptr;
    ws->bytes = 0;
    ws->retired.clear();
  }
  g_workspaces.clear();
  if (have_dev) (void)hipSetDevice(cur);
  return rc;
}

}  // extern "C"
