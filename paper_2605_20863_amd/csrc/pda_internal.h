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

enum class KvType : int { F32 = 0, BF16 = 1, FP8 = 2 };
enum class Variant : int { Vector = 1, Mfma = 2 };

// Device-side status bits (workspace header word kHdrStatus).
constexpr int kStatusLenClamped = 1;
constexpr int kStatusBadBlock = 2;

// Workspace header words.
constexpr int kHdrStatus = 0;
constexpr int kHdrShare = 1;  // block-heads per chunk (decode writes, combine reads)
constexpr int kHdrNext = 2;   // chunk counter of a dynamic split; zero between calls
constexpr int kHdrWords = 16;

// Everything one decode step's kernels need. Plain data; passed by value.
struct DecodeArgs {
  const void* q;
  const void* k_cache;
  const void* v_cache;
  const int32_t* block_table;
  const int32_t* seq_lens;
  const float* kv_scales;
  void* out;
  float scale_log2;     // softmax_scale * log2(e): logits are kept in base 2
  int32_t B, Hq, Hkv, G, D;
  int32_t max_blocks;   // block_table row stride
  int64_t num_blocks;   // physical blocks (for the bounds check of table entries)
  int32_t len_cap;      // lengths are clamped into [0, len_cap]
  int32_t min_share;    // smallest chunk, in block-heads
  int32_t chunk_min;    // a dynamic split makes no chunk smaller than this
  int32_t chunks_max;   // at most this many chunks; <= waves means a static split
  int32_t waves;        // launched persistent waves (a multiple of waves_per_group)
  int32_t waves_per_group;  // independent stream-K waves per workgroup: 1, 2 or 4
  int32_t out_bf16;     // 1: out is bf16, 0: f32
  // workspace
  int32_t* hdr;         // kHdrWords ints
  int32_t* cum;         // [B] exclusive prefix sum of blocks per sequence
  int32_t* share;       // [1] block-heads per chunk (written by wave 0, read by the combine)
  float* ws_m;          // [slots, G] running max (base 2) per partial
  float* ws_l;          // [slots, G] softmax denominator per partial
  float* ws_acc;        // [slots, G, D] unnormalised output per partial
};

// Number of partial-result slots one call can need: one per (unit, chunk)
// intersection, bounded by units + chunks.
inline int64_t partial_slots(int B, int Hkv, int chunks_max) {
  return (int64_t)B * Hkv + chunks_max;
}

// Launchers (pda_kernels.hip). Return hipSuccess or the launch error.
hipError_t launch_decode(const DecodeArgs& a, Variant v, KvType kv, hipStream_t s);
hipError_t launch_combine(const DecodeArgs& a, hipStream_t s);
// Max resident waves per CU for the decode kernel that (v, kv, D, G) selects.
hipError_t decode_occupancy(Variant v, KvType kv, int D, int G, int* waves_per_cu);

}  // namespace pda
