// Internal interface between the C-ABI host code (pda_host.cpp) and the HIP
// kernels (pda_kernels.hip). Not installed; callers use include/pda.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pda {

constexpr int kBlockSize = 16;     // tokens per KV block
constexpr int kWave = 64;          // CDNA wavefront width
constexpr int kMaxGroup = 16;      // query heads per KV head (MFMA N dimension)
constexpr int kMaxGroupVector = 8; // vector kernel keeps G x D/16 query values per lane
constexpr int kWideColumns = 32;   // query columns of a wide entry (two MFMA N-tiles)
// The stream-K split cuts a stream in which every block-head is one unit of
// work and every (entry, KV head) with blocks costs this many more before its
// first block: a wave's fixed cost of starting a segment (query loads, the
// load pipeline filling, the partial's write; about two block-heads' time for
// a one-tile segment, more for a two-tile one with twice the query columns
// and partial), so waves whose chunks cross many short units get fewer
// blocks. In shared-prefix mode and in plain mode.
constexpr int kUnitCostShared = 4;
constexpr int kUnitCostPlain = 2;

enum class KvType : int { F32 = 0, BF16 = 1, FP8 = 2 };
enum class Variant : int { Vector = 1, Mfma = 2 };

// Device-side status bits (workspace header word kHdrStatus).
constexpr int kStatusLenClamped = 1;
constexpr int kStatusBadBlock = 2;
constexpr int kStatusPrefixShortened = 4;  // a group's members share fewer leading blocks than declared
constexpr int kStatusBadOffsets = 8;       // prefill: q_offsets not non-decreasing within [0, T]
constexpr int kStatusHalfRange = 16;       // prefill: a V value outside the fp16 range was saturated

// Workspace header words.
constexpr int kHdrStatus = 0;
constexpr int kHdrShare = 1;  // block-heads per chunk (decode writes, combine reads)
constexpr int kHdrNext = 2;   // chunk counter of a dynamic split; zero between calls
constexpr int kHdrItems = 3;  // prefill: work items the plan kernel listed
constexpr int kHdrPfQueue = 8;  // prefill: words 8..15, the unit counters of the attention grid's queues
constexpr int kHdrWords = 16;

// Everything one decode step's kernels need. Plain data; passed by value.
// The decode kernels keep it in registers; two more int32 fields once made
// the compiler place the whole struct in scratch memory (248 bytes per lane,
// every kernel), so a new field is worth checking with the resource-usage
// remarks.
struct DecodeArgs {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const float* kv_scales;
  void* out;
  float scale_log2;     // softmax_scale * log2(e): logits are kept in base 2
  float mfma_scale_log2; // |softmax_scale| * log2(e): the MFMA body flips q's sign for a negative scale
  int32_t neg_scale;    // 1: softmax_scale < 0
  int32_t B, Hq, Hkv, G, D;
  int32_t max_blocks;   // block_table row stride
  int64_t num_blocks;   // physical blocks (for the bounds check of table entries)
  int32_t len_cap;      // lengths are clamped into [0, len_cap]
  int32_t min_share;    // smallest chunk, in stream units (block-heads plus unit start costs)
  int32_t chunk_min;    // a dynamic split makes no chunk smaller than this
  int32_t chunks_max;   // at most this many chunks; <= waves means a static split
  int32_t waves;        // launched persistent waves (a multiple of waves_per_group)
  int32_t waves_per_group;  // independent stream-K waves per workgroup: 1, 2 or 4
  int32_t out_bf16;     // 1: out is bf16, 0: f32
  int32_t Qn;           // query tokens per sequence: q and out are [B, Qn, Hq, D]
  // Work entries. Plain mode: entry b is sequence b (E = B). Shared-prefix
  // mode: entries [0, n_prefix) are the groups' shared leading blocks, nsub
  // per group, each applied to the queries of up to M members (M * G query
  // columns); entry n_prefix + m is the rest of sequence m.
  int32_t E;
  int32_t shared;       // 1: shared-prefix mode
  int32_t group_size;   // members per group (sequences g * group_size ..)
  int32_t M;            // members per prefix entry (M * G <= kWideColumns)
  int32_t nsub;         // prefix entries per group = ceil(group_size / M)
  int32_t n_prefix;     // num_groups * nsub
  int32_t Gp;           // query columns per partial row: Qn * G, or M * G in shared-prefix mode
  const int32_t* shared_blocks;  // [num_groups] caller's bound on each group's shared blocks
  // workspace
  int32_t* hdr;         // kHdrWords ints
  int32_t* sg;          // [num_groups] shared blocks each group really has (prefix kernel)
  int32_t* cum;         // [E] exclusive prefix sum of blocks per entry
  int32_t* share;       // [1] block-heads per chunk (written by wave 0, read by the combine)
  float* ws_m;          // [slots, Gp] running max (base 2) per partial
  float* ws_l;          // [slots, Gp] softmax denominator per partial
  float* ws_acc;        // [slots, Gp, D] unnormalised output per partial
};

// Number of partial-result slots one call can need: one per (unit, chunk)
// intersection, bounded by units + chunks (a unit is an (entry, KV head)).
inline int64_t partial_slots(int64_t entries, int Hkv, int chunks_max) {
  return entries * Hkv + chunks_max;
}

// One step's KV append (pda_append.hip).
struct AppendArgs {
  const void* k_new;    // [B, Hkv, D] f32 or bf16
  const void* v_new;
  void* k_cache;        // [NB, Hkv, 16, D]
  void* v_cache;        // [NB, Hkv, D, 16]
  float* kv_scales;     // [2, NB, Hkv] (fp8 caches)
  const int32_t* block_table;
  const int32_t* positions;  // [B] slot of the new token; < 0 skips the sequence
  int32_t B, Hkv, D, max_blocks;
  int64_t num_blocks;
  int32_t new_bf16;     // 1: k_new / v_new are bf16, 0: f32
  int32_t* status;      // workspace status word
};

hipError_t launch_append(const AppendArgs& a, KvType kv, hipStream_t s);

// Variable-length causal prefill (pda_prefill.hip).
constexpr int kPfColumns = 256;  // query (token, head) columns per workgroup
constexpr int kPfBuckets = 2048; // length classes of the plan's counting sort

struct PrefillArgs {
  const void* q;        // [T, Hq, D] bf16
  const int32_t* q_offsets;  // [B + 1]
  const void* k_cache;
  const void* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const float* kv_scales;
  void* out;            // [T, Hq, D] bf16 or f32
  float scale_log2;     // |softmax_scale| * log2(e)
  int32_t neg_scale;    // 1: softmax_scale < 0 (q enters with its sign flipped)
  int32_t B, T, Hq, Hkv, G, D;
  int32_t TQ;           // query tokens per tile: kPfColumns / G
  int32_t max_blocks;
  int64_t num_blocks;
  int32_t len_cap;
  int32_t len_shift;    // sort key: length >> len_shift, below kPfBuckets
  int32_t items_max;    // bound on the work items (units: items x KV heads)
  int32_t out_bf16;
  int32_t cus;          // compute units of the device
  int32_t nq;           // unit queues: gcd(Hkv, 8)
  int32_t* hdr;         // workspace header (status, item count, queue counters)
  int4* items;          // [items_max] {sequence, first q row, tokens, first position}
  // Image of the cache's tiles in the products' operand types, indexed like the
  // cache (block * Hkv + KV head, 16 * D two-byte elements per tile): V in fp16
  // (v_img), and for an fp8 cache K in bf16 (k_img). v_img null: the attention
  // kernel stages the tiles through registers instead.
  void* k_img;
  void* v_img;
};

hipError_t launch_prefill(const PrefillArgs& a, KvType kv, hipStream_t s);

// Launchers (pda_kernels.hip). Return hipSuccess or the launch error.
hipError_t launch_decode(const DecodeArgs& a, Variant v, KvType kv, hipStream_t s);
hipError_t launch_combine(const DecodeArgs& a, hipStream_t s);
// Shared-prefix mode: the groups' real shared block counts, before the decode kernel.
hipError_t launch_prefix(const DecodeArgs& a, int num_groups, hipStream_t s);
// Fixed device scratch of pda_paged_decode_attention_noalloc: a file-scope
// array in pda_scratch.hip, one copy per device, used in place of the
// stream's workspace (same layout). 32 MiB holds the workspace of every
// decode step up to 512 sequences x 8 KV heads x 32 query columns at the
// default split (about 25 MiB for the fp8 step at 64 / 8 heads).
constexpr int64_t kScratchBytes = 32ll << 20;
// Device address of the current device's copy of that array
// (hipGetSymbolAddress; the caller keeps it per device).
hipError_t scratch_address(void** ptr);

// Max resident waves per CU for the decode kernel that (v, kv, D, G) selects.
// wide: the kernel whose entries carry up to kWideColumns query columns (shared-prefix
// prefix entries, several query tokens per sequence)
hipError_t decode_occupancy(Variant v, KvType kv, int D, int G, bool wide, int* waves_per_cu);

}  // namespace pda
