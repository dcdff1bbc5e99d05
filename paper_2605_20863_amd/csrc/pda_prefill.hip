// HIP kernels for variable-length causal prefill over the paged KV cache on
// MI355X (gfx950, CDNA4).
//
// The log-prob forward of RLVR training (the compute_log_prob phase timed in
// the paper's Table 2, Sec. 6.3; a forward call of its Sec. 4.2 interface) and
// chunked prefill attend many query tokens per sequence at once: packed q rows
// q_offsets[b] .. q_offsets[b+1]-1 are the last n_b of sequence b's L_b cached
// tokens, and token i (position L_b - n_b + i) sees tokens 0 .. L_b - n_b + i.
// This is compute-bound: every K and V element is reused by all query columns
// of a tile, so K and V go through LDS once per workgroup and the products run
// on the matrix cores.
//
// * Prep kernel. Workgroup 0 plans: per sequence, its tiles of 256 / G query
//   tokens; sequences sorted by length, longest first (counting sort on the
//   length), and a work list of (sequence, tile) items, each sequence's last
//   (heaviest) tile first. The other workgroups (image path) write the image:
//   every tile of a block that a sequence with queries reads, converted to the
//   operand types of the products (V to fp16, fp8 as code times the block's V
//   scale; for fp8 caches K codes to bf16), indexed like the cache.
// * Attention kernel: a persistent grid, one workgroup (8 waves, 2 per SIMD)
//   per CU, that takes (item, KV head) units from queues, so a CU goes from one
//   unit to the next without a workgroup launch between them (which cost ~4 us
//   per unit, with the drain of the last workgroup's waves). There are
//   nq = gcd(Hkv, 8) queues; queue x holds the units of KV heads x, x + nq, ...
//   in item order, and workgroup i works on queue (i % 8) % nq. The dispatcher
//   deals workgroups round-robin over the 8 XCDs, so with 4 or 8 KV heads each
//   XCD serves one KV head and its L2 holds only that head's keys and values,
//   read by every tile of a sequence at nearly the same time (a drained queue
//   sends its workgroups to the others; correctness never depends on the XCD).
//   A unit's query columns are (token, head) pairs, 256 / G tokens times the G
//   query heads of the KV head; each wave owns 32 columns (2 MFMA N-tiles).
// * The KV prefix up to the tile's last position is walked two 16-token blocks
//   (32 keys, a pair) at a time, two pairs per barrier, from four LDS buffers:
//   while a step computes two pairs, the next two pairs' tiles travel to the
//   other two buffers. On the image path they go straight from memory to LDS
//   (global_load_lds, two 16-byte pieces per lane and pair, no registers and
//   no conversion instructions); on the staging path (an image larger than the
//   host allows) each thread loads its pieces into registers, converts them and
//   writes them to LDS between the step's two pairs.
// * Key order: lane group c (lanes 16c .. 16c + 15) holds keys 8c .. 8c + 7 of
//   a pair in its score and P^T registers, 8 consecutive tokens of one block,
//   so a 16-byte V operand is one 16-byte piece of a cached dim row.
// * Per wave and pair: S^T[32 keys x 32 columns] = K . Q^T on
//   v_mfma_f32_16x16x32_bf16, online softmax on the accumulators (lazy
//   rescale), weights packed to fp16 and O^T += V^T . P^T on
//   v_mfma_f32_16x16x32_f16; the row sums come from a product with a ones
//   operand, so they add exactly the fp16 weights the product uses. The K scale
//   of an fp8 block goes on its logits. LDS operand reads sit beside matrix
//   work: the second pair of a step has its K operands read between the first
//   pair's P . V MFMAs, and every pair its V operands between its own score
//   MFMAs (on the staging path, where the staged registers are still live
//   then, the first pair reads half of them during its softmax instead).
// * Causal masking selects per column (a key is seen iff it is at or before the
//   column's position); V rows of keys past the tile's last position are zeroed,
//   so NaN poison in unused slots never reaches the products. Only pairs that
//   reach past a wave's first position take the masked path, and a wave skips
//   the pairs past its last position.

#include "pda_internal.h"

#include <stdint.h>

#include <atomic>
#include <type_traits>

namespace pda {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kPfWaves = 8;
constexpr int kPfThreads = 64 * kPfWaves;
constexpr int kPfNT = 2;                // 16-column N-tiles per wave
constexpr int kPfWaveCols = 16 * kPfNT; // query columns per wave
constexpr float kNegInf = -__builtin_inff();
constexpr float kSlack = 8.f;  // lazy-rescale slack (log2 units): weights stay below 2^8
constexpr int kPlanThreads = 1024;
static_assert(kPfWaves * kPfNT * 16 == kPfColumns, "columns per workgroup");
static_assert(kPfBuckets % kPlanThreads == 0, "buckets per plan thread");

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t w) {
  u32x2 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, false));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, true));
  return r;
}

// codes 0, 1 (HI false) or 2, 3 (HI true) of a word of four E4M3 codes, times
// scale (the conversion's own scale operand is a power-of-two exponent, so the
// tile scale is applied in fp32 afterwards)
template <bool HI>
__device__ __forceinline__ float2 fp8x2_to_f32x2(uint32_t w, float scale) {
  const f32x2 v = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8((int)w, 1.0f, HI);
  return float2{v.x * scale, v.y * scale};
}

__device__ __forceinline__ uint32_t pk_f16(float x, float y) {
  f16x2 h;
  h[0] = (_Float16)x;
  h[1] = (_Float16)y;
  return __builtin_bit_cast(uint32_t, h);
}

// two f32 -> packed bf16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint32_t pk_bf16(float x, float y) {
  bf16x2 h;
  h[0] = (__bf16)x;
  h[1] = (__bf16)y;
  return __builtin_bit_cast(uint32_t, h);
}

// ------------------------------------------------------------------ plan

struct PfSeq {
  int q0, n, L, tiles, key;
};

// Sequence b as the plan sees it: lengths are clamped into [0, len_cap]
// (status bit 1); `bad` is set when its offsets leave [0, T] or decrease. key
// orders sequences longest first.
__device__ PfSeq pf_seq(const PrefillArgs& a, int b, int& status, bool& bad) {
  PfSeq s;
  const int o0 = a.q_offsets[b], o1 = a.q_offsets[b + 1];
  s.q0 = o0;
  s.n = o1 - o0;
  if (o0 < 0 || o1 > a.T || o1 < o0) {
    bad = true;
    s.n = 0;
  }
  int L = a.seq_lens[b];
  if (L > a.len_cap || L < 0) {
    status |= kStatusLenClamped;
    L = L < 0 ? 0 : a.len_cap;
  }
  s.L = L;
  s.tiles = (s.n + a.TQ - 1) / a.TQ;
  const int k = L >> a.len_shift;
  s.key = kPfBuckets - 1 - (k < kPfBuckets - 1 ? k : kPfBuckets - 1);
  return s;
}

// Offsets that are not non-decreasing within [0, T] list no item at all (status
// bit 8): with them the sequences could overlap and overrun the list. Otherwise
// the tiles add up to at most (T + B (TQ - 1)) / TQ = items_max.
__device__ void pf_plan(const PrefillArgs& a) {
  __shared__ int cursor[kPfBuckets];
  __shared__ int wave_sum[kPlanThreads / 64];
  const int tid = (int)threadIdx.x;
  for (int i = tid; i < kPfBuckets; i += kPlanThreads) cursor[i] = 0;
  if (tid < 8) a.hdr[kHdrPfQueue + tid] = 0;
  __syncthreads();
  int status = 0;
  bool bad = false;
  for (int b = tid; b < a.B; b += kPlanThreads) {
    const PfSeq s = pf_seq(a, b, status, bad);
    if (s.tiles) atomicAdd(&cursor[s.key], s.tiles);
  }
  if (__syncthreads_or(bad)) {
    if (tid == 0) {
      a.hdr[kHdrItems] = 0;
      atomicOr(a.hdr + kHdrStatus, kStatusBadOffsets);
    }
    return;
  }
  // exclusive scan of the per-bucket tile counts: bucket starts in the list
  constexpr int PER = kPfBuckets / kPlanThreads;
  int v[PER], run = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    v[i] = cursor[tid * PER + i];
    run += v[i];
  }
  int x = run;
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const int y = __shfl_up(x, o, 64);
    if (l >= o) x += y;
  }
  if (l == 63) wave_sum[tid >> 6] = x;
  __syncthreads();
  int before = 0;
  for (int w = 0; w < (tid >> 6); ++w) before += wave_sum[w];
  int start = before + x - run;
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    cursor[tid * PER + i] = start;
    start += v[i];
  }
  if (tid == kPlanThreads - 1) a.hdr[kHdrItems] = start;  // total items
  __syncthreads();
  for (int b = tid; b < a.B; b += kPlanThreads) {
    const PfSeq s = pf_seq(a, b, status, bad);
    if (!s.tiles) continue;
    int pos = atomicAdd(&cursor[s.key], s.tiles);
    for (int t = s.tiles - 1; t >= 0; --t) {  // the last (heaviest) tile first
      const int t0 = t * a.TQ;
      const int nt = s.n - t0 < a.TQ ? s.n - t0 : a.TQ;
      a.items[pos++] = make_int4(b, s.q0 + t0, nt, s.L - s.n + t0);
    }
  }
  if (status) atomicOr(a.hdr + kHdrStatus, status);
}

// ------------------------------------------------------- layout and image

// LDS layout of one pair (two 16-token blocks of one KV head), the same on both
// paths:
//   K [32 keys][D] bf16 (fp8: the codes, exact in bf16); the 16-byte chunk h
//     of key row k sits at chunk h ^ kswz(k), so the 16 rows that one K operand
//     read touches fall on distinct banks
//   V [2 blocks][D dims][16 tokens] fp16 (fp8: code * V scale); the 8-token
//     half h of dim row d sits at half h ^ ((d >> 3) & 1)
// Image tiles keep the cache's own layout (K [16 tokens][D] bf16, V [D][16
// tokens] fp16), so a direct load copies 16-byte pieces of a tile.
template <KvType KV, int D>
struct PfCfg {
  static constexpr int GSZ = KV == KvType::FP8 ? 1 : 2;  // bytes per cached element
  static constexpr int KSTEPS = D / 32;                 // 16x16x32 k-steps over head_dim
  static constexpr int MT = D / 16;                     // 16-row tiles of O^T
  static constexpr int GTILE = 16 * D * GSZ;            // bytes of one cached (block, KV head) tile
  static constexpr int TILEB = 16 * D * 2;              // bytes of one image tile (and of a bf16 cache tile)
  static constexpr int KROW = 2 * D;                    // bytes of an LDS K row
  static constexpr int KBUF = 32 * KROW;
  static constexpr int VBLK = 32 * D;                   // bytes of one block's V part in LDS
  static constexpr int BUF = KBUF + 2 * VBLK;
  static constexpr int NI = D / 64;                     // direct loads per wave and pair
  // staging unit: 8 elements (16 bytes of bf16, 8 bytes of fp8), so fp8 pairs keep every thread busy
  static constexpr int UB = 8 * GSZ;
  static constexpr int UNITS = 2 * GTILE / UB;          // units of a pair's K (or V) tiles
  static constexpr int UPT = (UNITS + kPfThreads - 1) / kPfThreads;
};

template <int D>
__device__ __forceinline__ int pf_kswz(int k) {
  if constexpr (D == 128) return (k & 3) | ((k >> 3) << 2);
  else return ((k >> 1) & 1) | ((k >> 3) << 1);
}

constexpr float kHalfMax = 65504.f;  // largest finite fp16

// V values (f32) -> packed fp16 pairs. Values within the fp16 range convert
// as they are; larger ones saturate, and `ovf` records one whose key is live
// (poison in a dead slot does not count).
template <int N>
__device__ __forceinline__ void v_pack(const float (&f)[N], uint32_t (&out)[N / 2], int k0, int live, int& ovf) {
  float amax = 0.f;
#pragma unroll
  for (int i = 0; i < N; ++i) amax = fmaxf(amax, fabsf(f[i]));
  if (amax > kHalfMax) {
#pragma unroll
    for (int i = 0; i < N; ++i) ovf |= k0 + i < live && fabsf(f[i]) > kHalfMax;
#pragma unroll
    for (int i = 0; i < N / 2; ++i)
      out[i] = pk_f16(__builtin_amdgcn_fmed3f(f[2 * i], -kHalfMax, kHalfMax),
                      __builtin_amdgcn_fmed3f(f[2 * i + 1], -kHalfMax, kHalfMax));
  } else {
#pragma unroll
    for (int i = 0; i < N / 2; ++i) out[i] = pk_f16(f[2 * i], f[2 * i + 1]);
  }
}

// 8 bf16 (one 16-byte piece) -> 8 fp16; k0: key index of the first, live: keys that exist
__device__ __forceinline__ u32x4 bf16x8_to_half(u32x4 x, int k0, int live, int& ovf) {
  float f[8];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __builtin_bit_cast(float, x[i] << 16);
    f[2 * i + 1] = __builtin_bit_cast(float, x[i] & 0xFFFF0000u);
  }
  uint32_t h[4];
  v_pack<8>(f, h, k0, live, ovf);
  return u32x4{h[0], h[1], h[2], h[3]};
}

// 8 E4M3 codes times the block's V scale -> 8 fp16, one rounding from fp32
__device__ __forceinline__ u32x4 fp8x8_to_half(u32x2 x, float vs, int k0, int live, int& ovf) {
  float f[8];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const float2 x01 = fp8x2_to_f32x2<false>(x[i], vs), x23 = fp8x2_to_f32x2<true>(x[i], vs);
    f[4 * i] = x01.x;
    f[4 * i + 1] = x01.y;
    f[4 * i + 2] = x23.x;
    f[4 * i + 3] = x23.y;
  }
  uint32_t h[4];
  if (vs * 448.f <= kHalfMax) {  // no code can leave the fp16 range
#pragma unroll
    for (int i = 0; i < 4; ++i) h[i] = pk_f16(f[2 * i], f[2 * i + 1]);
  } else {
    v_pack<8>(f, h, k0, live, ovf);
  }
  return u32x4{h[0], h[1], h[2], h[3]};
}

// 8 E4M3 codes -> 8 bf16 (exact, unscaled: the K scale goes on the logits)
__device__ __forceinline__ u32x4 fp8x8_to_bf16(u32x2 x) {
  const u32x2 a0 = fp8x4_to_bf16x4(x.x), a1 = fp8x4_to_bf16x4(x.y);
  return u32x4{a0.x, a0.y, a1.x, a1.y};
}

constexpr int kImgBlocks = 16;  // table entries per image workgroup
constexpr int kImgBatch = 4;    // pieces a thread loads before it converts and stores them

// Image workgroup g: table entries kImgBlocks * (g % cps) + 0 .. kImgBlocks - 1
// of sequence g / cps. Every tile (all KV heads) of a block that a sequence
// with queries reads, keys 0 .. L_b - 1, is converted to the image, indexed
// like the cache (block * Hkv + KV head); blocks shared by several sequences
// are written by each with the same bytes. Entries outside [0, num_blocks) are
// skipped (the attention kernel flags them). A live V value beyond the fp16
// range saturates and sets status bit 16.
template <KvType KV, int D>
__device__ void pf_image(const PrefillArgs& a, int g) {
  using C = PfCfg<KV, D>;
  const int cps = (a.max_blocks + kImgBlocks - 1) / kImgBlocks;
  const int b = g / cps;
  const int j0 = (g - b * cps) * kImgBlocks;
  const int o0 = a.q_offsets[b], o1 = a.q_offsets[b + 1];
  if (o0 < 0 || o1 > a.T || o1 <= o0) return;  // no queries, or offsets the plan rejects
  int L = a.seq_lens[b];
  L = L < 0 ? 0 : (L > a.len_cap ? a.len_cap : L);
  const int nblk = (L + 15) / 16;
  const int nb = nblk - j0 < kImgBlocks ? nblk - j0 : kImgBlocks;
  if (nb <= 0) return;
  // a piece is 16 bytes of the cache: 8 bf16 values, or 16 fp8 codes (for V a
  // whole dim row of the block, for K 16 dims of one token)
  constexpr int EPP = KV == KvType::FP8 ? 16 : 8;  // elements per piece
  constexpr int UT = 16 * D / EPP;                 // pieces of a tile
  const int vpieces = a.Hkv * UT;
  const int per_blk = KV == KvType::FP8 ? 2 * vpieces : vpieces;  // fp8: V pieces, then K pieces
  const int total = nb * per_blk;
  const int32_t* row = a.block_table + (int64_t)b * a.max_blocks;
  const uint8_t* kc = static_cast<const uint8_t*>(a.k_cache);
  const uint8_t* vc = static_cast<const uint8_t*>(a.v_cache);
  uint8_t* ki = static_cast<uint8_t*>(a.k_img);
  uint8_t* vi = static_cast<uint8_t*>(a.v_img);
  int ovf = 0;
  for (int u0 = (int)threadIdx.x; u0 < total; u0 += kImgBatch * kPlanThreads) {
    u32x4 x[kImgBatch];
    int64_t tile[kImgBatch];
    int e[kImgBatch], live[kImgBatch], kind[kImgBatch];  // kind: 0 none, 1 V, 2 K
    float vs[kImgBatch];
#pragma unroll
    for (int i = 0; i < kImgBatch; ++i) {
      const int u = u0 + i * kPlanThreads;
      kind[i] = 0;
      if (u >= total) continue;
      const int jj = u / per_blk;
      int rest = u - jj * per_blk;
      const int p = row[j0 + jj];
      if ((uint64_t)(uint32_t)p >= (uint64_t)a.num_blocks) continue;
      const bool is_k = rest >= vpieces;
      if (is_k) rest -= vpieces;
      const int h = rest / UT;
      e[i] = rest - h * UT;
      tile[i] = (int64_t)p * a.Hkv + h;
      live[i] = L - 16 * (j0 + jj);
      kind[i] = is_k ? 2 : 1;
      x[i] = *reinterpret_cast<const u32x4*>((is_k ? kc : vc) + tile[i] * C::GTILE + e[i] * 16);
      vs[i] = 1.f;
      if constexpr (KV == KvType::FP8) {
        if (!is_k) vs[i] = a.kv_scales[a.num_blocks * a.Hkv + tile[i]];
      }
    }
#pragma unroll
    for (int i = 0; i < kImgBatch; ++i) {
      if (kind[i] == 0) continue;
      uint8_t* dst = (kind[i] == 2 ? ki : vi) + tile[i] * C::TILEB + e[i] * (2 * EPP);
      if constexpr (KV == KvType::FP8) {
        const u32x2 lo{x[i].x, x[i].y}, hi{x[i].z, x[i].w};
        if (kind[i] == 2) {  // K: 16 dims of one token
          *reinterpret_cast<u32x4*>(dst) = fp8x8_to_bf16(lo);
          *reinterpret_cast<u32x4*>(dst + 16) = fp8x8_to_bf16(hi);
        } else {             // V: dim row e, tokens 0 .. 15
          *reinterpret_cast<u32x4*>(dst) = fp8x8_to_half(lo, vs[i], 0, live[i], ovf);
          *reinterpret_cast<u32x4*>(dst + 16) = fp8x8_to_half(hi, vs[i], 8, live[i], ovf);
        }
      } else {  // V piece e: dim row e / 2, tokens 8 (e % 2) .. + 7
        *reinterpret_cast<u32x4*>(dst) = bf16x8_to_half(x[i], 8 * (e[i] & 1), live[i], ovf);
      }
    }
  }
  if (ovf) atomicOr(a.hdr + kHdrStatus, kStatusHalfRange);
}

__global__ __launch_bounds__(kPlanThreads) void prefill_plan_kernel(PrefillArgs a) { pf_plan(a); }

// The plan (workgroup 0) and the image (the others) in one launch.
template <KvType KV, int D>
__global__ __launch_bounds__(kPlanThreads) void prefill_prep_kernel(PrefillArgs a) {
  if (blockIdx.x == 0) {
    pf_plan(a);
    return;
  }
  pf_image<KV, D>(a, (int)blockIdx.x - 1);
}

// ------------------------------------------------------------- attention

// The tile's physical block ids, 64 at a time: lane i holds the id of block
// 64q + i of chunk q, read with one vector load per chunk, the next chunk's
// ids one chunk ahead, so a pair's ids come from v_readlane instead of a
// scalar load per block.
struct PfIds {
  int q;          // current chunk
  int id, nxt;    // table entries of chunks q and q + 1, unchecked (lanes past the tile repeat its last block)
};

// Unconditional, and checked only where a pair reads it (pf_pair): a check
// here would wait for the load at once and the next chunk would not be
// prefetched. The table row has max_blocks >= 1 entries and nblk <= max_blocks.
__device__ __forceinline__ int pf_id_load(const int32_t* row, int j, int nblk) {
  const int last = nblk > 0 ? nblk - 1 : 0;
  return row[j < last ? j : last];
}

// Moves the ids to chunk q (q is ids.q or ids.q + 1) and loads chunk q + 1.
// Unconditional: no loaded register is merged across paths (a copy of one
// waits for its load), and the select reads a load issued a step earlier.
__device__ __forceinline__ void pf_ids_advance(PfIds& ids, const int32_t* row, int q, int nblk) {
  ids.id = q != ids.q ? ids.nxt : ids.id;
  ids.q = q;
  ids.nxt = pf_id_load(row, 64 * (q + 1) + lane_id(), nblk);
}

__device__ __forceinline__ int64_t uni64(int64_t x) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)x);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)((uint64_t)x >> 32));
  return (int64_t)(((uint64_t)hi << 32) | lo);
}

// One pair's blocks, workgroup-uniform: tiles (block * Hkv + KV head; a block
// with no id names tile 0 of its KV head, whose keys are masked), flags,
// fp8 scales as loaded (used only after the next wait) and live keys. Named
// fields, not two-element arrays: a select between array elements can become
// an indexed access, which puts the array in scratch memory.
struct PfPair {
  int64_t t0, t1;
  int ok0, ok1;   // block holds keys of the tile and its id is in range
  float ks0, ks1, vs0, vs1;
  int live;       // keys of the pair that exist (from the pair's first key)
};

template <KvType KV, bool IMG>
__device__ __forceinline__ PfPair pf_pair(const PrefillArgs& a, const PfIds& ids, int j0, int nblk, int nkeys,
                                          int kvh, int& status) {
  int64_t tile[2];
  int ok[2];
  float ks[2] = {1.f, 1.f}, vs[2] = {1.f, 1.f};
  // ids are int32: p is a block iff 0 <= p < num_blocks, one unsigned 32-bit
  // compare against min(num_blocks, 2^31) (scalar: there is no 64-bit scalar <)
  const uint32_t nbu = a.num_blocks < (1ll << 31) ? (uint32_t)a.num_blocks : 0x80000000u;
#pragma unroll
  for (int s = 0; s < 2; ++s) {
    const int p = __builtin_amdgcn_readlane(ids.id, (j0 + s) & 63);
    const bool inside = j0 + s < nblk;  // the block holds keys of the tile
    ok[s] = inside && (uint32_t)p < nbu;
    if (inside && !ok[s]) status |= kStatusBadBlock;
    tile[s] = uni64((int64_t)(ok[s] ? p : 0) * a.Hkv + kvh);
    if constexpr (KV == KvType::FP8) {  // raw: a block with no id takes scale 1 where they are used
      ks[s] = a.kv_scales[tile[s]];
      if constexpr (!IMG) vs[s] = a.kv_scales[a.num_blocks * a.Hkv + tile[s]];
    }
  }
  int live = nkeys - 16 * j0;
  if (!ok[1]) live = live < 16 ? live : 16;
  if (!ok[0]) live = 0;
  return PfPair{tile[0], tile[1], ok[0], ok[1], ks[0], ks[1], vs[0], vs[1], live};
}

// V scale of block s of the pair (1 for a block with no id; staging path)
__device__ __forceinline__ float pf_vs(const PfPair& pp, int s) {
  return s ? (pp.ok1 ? pp.vs1 : 1.f) : (pp.ok0 ? pp.vs0 : 1.f);
}

// Per-pair values a wave needs once the pair's tiles are in LDS.
struct PfMeta {
  float c0, c1;  // softmax scale (log2 units) times the blocks' K scales, > 0
  int live;      // keys of the pair that exist
};

__device__ __forceinline__ PfMeta pf_meta(const PfPair& pp, float scale_log2) {
  // c > 0: a zero or tiny scale leaves every weight at 1 either way
  const float k0 = pp.ok0 ? pp.ks0 : 1.f, k1 = pp.ok1 ? pp.ks1 : 1.f;
  return PfMeta{fmaxf(scale_log2 * k0, 1e-30f), fmaxf(scale_log2 * k1, 1e-30f), pp.live};
}

// ---- image path: direct loads

// A wave's part of a pair's direct loads: per load, K or V, which of the two
// blocks, this lane's byte offset in that block's tile, and the LDS offset in
// the pair's buffer of the load's first lane (lane i writes 16 bytes at + 16 i).
template <int D>
struct PfLane {
  int is_v[D / 64], blk[D / 64], dst[D / 64];
  uint32_t off[D / 64];
};

// D = 128: wave w loads K rows 4w .. 4w + 3 (block w / 4) and V dim rows
// 32 (w % 4) .. + 31 of block w / 4. D = 64: waves 0-3 load K rows 8w .. 8w + 7,
// waves 4-7 V dim rows 32 (w % 2) .. + 31 of block (w - 4) / 2.
template <int D>
__device__ __forceinline__ PfLane<D> pf_lane(int w, int l) {
  PfLane<D> pl;
  const int kbuf = 32 * 2 * D;
  if constexpr (D == 128) {
    const int row = 4 * w + (l >> 4);
    pl.is_v[0] = 0;
    pl.blk[0] = w >> 2;
    pl.dst[0] = 1024 * w;
    pl.off[0] = (uint32_t)((row & 15) * 256 + 16 * ((l & 15) ^ pf_kswz<D>(row)));
    const int d = 32 * (w & 3) + (l >> 1);
    pl.is_v[1] = 1;
    pl.blk[1] = w >> 2;
    pl.dst[1] = kbuf + 1024 * w;
    pl.off[1] = (uint32_t)(d * 32 + 16 * ((l & 1) ^ ((d >> 3) & 1)));
  } else {
    if (w < 4) {
      const int row = 8 * w + (l >> 3);
      pl.is_v[0] = 0;
      pl.blk[0] = w >> 1;
      pl.dst[0] = 1024 * w;
      pl.off[0] = (uint32_t)((row & 15) * 128 + 16 * ((l & 7) ^ pf_kswz<D>(row)));
    } else {
      const int v = w - 4, d = 32 * (v & 1) + (l >> 1);
      pl.is_v[0] = 1;
      pl.blk[0] = v >> 1;
      pl.dst[0] = kbuf + 1024 * v;
      pl.off[0] = (uint32_t)(d * 32 + 16 * ((l & 1) ^ ((d >> 3) & 1)));
    }
  }
  return pl;
}

// One 16-byte piece per lane from base + off to LDS address lds + 16 * lane
// (global_load_lds_dwordx4; M0 holds the LDS address). base and lds are
// wave-uniform and made scalar here, as the instruction needs. The compiler
// does not see this load: completion is awaited with pf_dma_wait before the
// barrier that publishes the buffer. (Through the compiler's own builtin every
// LDS read in the kernel would wait for all LDS traffic, lgkmcnt(0).)
__device__ __forceinline__ void pf_dma16(const uint8_t* base_v, uint32_t off, uint32_t lds_v) {
  const uint8_t* base = reinterpret_cast<const uint8_t*>(uni64(reinterpret_cast<int64_t>(base_v)));
  const uint32_t lds = (uint32_t)__builtin_amdgcn_readfirstlane((int)lds_v);
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(off), "s"(base), "s"(lds) : "memory", "m0");
}
__device__ __forceinline__ void pf_dma_wait() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

template <KvType KV, int D>
__device__ __forceinline__ void pf_dma(const uint8_t* kimg, const uint8_t* vimg, int64_t t0, int64_t t1,
                                       const PfLane<D>& pl, uint32_t buf) {
  using C = PfCfg<KV, D>;
#pragma unroll
  for (int e = 0; e < C::NI; ++e) {
    const uint8_t* base = (pl.is_v[e] ? vimg : kimg) + (pl.blk[e] ? t1 : t0) * C::TILEB;
    pf_dma16(base, pl.off[e], buf + pl.dst[e]);
  }
}

// ---- staging path: registers

// One pair on its way to LDS: each thread's pieces of the cached K and V tiles.
template <KvType KV, int D>
struct PfStage {
  using Unit = typename std::conditional<KV == KvType::FP8, u32x2, u32x4>::type;
  Unit k[PfCfg<KV, D>::UPT], v[PfCfg<KV, D>::UPT];
};

template <KvType KV, int D>
__device__ __forceinline__ void pf_load(PfStage<KV, D>& st, const PrefillArgs& a, int64_t t0, int64_t t1) {
  using C = PfCfg<KV, D>;
  const uint8_t* kc = static_cast<const uint8_t*>(a.k_cache);
  const uint8_t* vc = static_cast<const uint8_t*>(a.v_cache);
  using Unit = typename PfStage<KV, D>::Unit;
  static_assert((C::GTILE / C::UB) % 64 == 0, "a wave's units lie in one block");
#pragma unroll
  for (int u = 0; u < C::UPT; ++u) {
    const int unit = (int)threadIdx.x + kPfThreads * u;
    const int blk = uni(unit / (C::GTILE / C::UB));  // the same for the whole wave
    const int off = (unit - blk * (C::GTILE / C::UB)) * C::UB;
    const int64_t base = (blk & 1 ? t1 : t0) * C::GTILE;  // uniform
    // Unconditional: a unit past the pair's tiles reads inside them (never
    // stored), so every path issues the same loads and the store that consumes
    // them waits for its own pair's loads only.
    st.k[u] = *reinterpret_cast<const Unit*>(kc + base + off);
    st.v[u] = *reinterpret_cast<const Unit*>(vc + base + off);
  }
}

template <KvType KV, int D>
__device__ __forceinline__ void pf_store(const PfStage<KV, D>& st, float vs0, float vs1, int live, uint8_t* buf,
                                         int& status) {
  using C = PfCfg<KV, D>;
  int ovf = 0;
#pragma unroll
  for (int u = 0; u < C::UPT; ++u) {
    const int unit = (int)threadIdx.x + kPfThreads * u;
    if (unit >= C::UNITS) break;
    const int blk = unit / (C::GTILE / C::UB);
    const int off = (unit - blk * (C::GTILE / C::UB)) * C::UB;
    const int krow = off / (D * C::GSZ), kh = (off - krow * D * C::GSZ) / (8 * C::GSZ);  // token row, chunk
    const int k = 16 * blk + krow;
    uint8_t* kdst = buf + k * C::KROW + 16 * (kh ^ pf_kswz<D>(k));
    const int d = off / (16 * C::GSZ), t0 = (off - d * 16 * C::GSZ) / C::GSZ;  // dim row, first token (0 or 8)
    uint8_t* vdst = buf + C::KBUF + blk * C::VBLK + d * 32 + 16 * ((t0 >> 3) ^ ((d >> 3) & 1));
    const int k0 = 16 * blk + t0;  // pair-relative key of token t0
    if constexpr (KV == KvType::BF16) {
      *reinterpret_cast<u32x4*>(kdst) = st.k[u];
      *reinterpret_cast<u32x4*>(vdst) = bf16x8_to_half(st.v[u], k0, live, ovf);
    } else {
      *reinterpret_cast<u32x4*>(kdst) = fp8x8_to_bf16(st.k[u]);
      *reinterpret_cast<u32x4*>(vdst) = fp8x8_to_half(st.v[u], blk & 1 ? vs1 : vs0, k0, live, ovf);
    }
  }
  if (ovf) status |= kStatusHalfRange;
}

// ---- per wave and pair

// Running softmax state of one 16-column N-tile (per lane: column r).
struct PfRow {
  float m;    // running max of the scaled logits (base 2); -inf before any key
  float nm;   // -m, or 0 while m = -inf: the exponent offset of the weights
  f32x4 l;    // sum of the fp16 weights (every row of a ones . P^T product)
};

// A pair's LDS operands in registers, one slot per K piece or V tile: slot i
// holds K piece i (d-step i / 2, t = i % 2), then V^T tile i (dim rows
// 16i + r). A pair's tiles replace its pieces, and the next pair's pieces
// replace the tiles.
template <KvType KV, int D>
struct PfOps {
  u32x4 x[PfCfg<KV, D>::MT];
};

// K piece i: lane (r, c) reads key row 8 (r / 4) + 4t + r % 4, d-step i / 2,
// so row 4c + e of the piece's scores is key 8c + 4t + e.
template <KvType KV, int D>
__device__ __forceinline__ void pf_kread(const uint8_t* buf, PfOps<KV, D>& o, int i) {
  using C = PfCfg<KV, D>;
  const int l = lane_id();
  const int r = l & 15, c = l >> 4;
  const int j = i >> 1, t = i & 1;
  const int k = 8 * (r >> 2) + 4 * t + (r & 3);
  o.x[i] = *reinterpret_cast<const u32x4*>(buf + k * C::KROW + 16 * ((4 * j + c) ^ pf_kswz<D>(k)));
}
// V tile m: lane (r, c) reads dim row 16m + r, keys 8c .. 8c + 7 (block c / 2,
// half c % 2), the P^T operand order.
template <KvType KV, int D>
__device__ __forceinline__ void pf_vread(const uint8_t* buf, PfOps<KV, D>& o, int m) {
  using C = PfCfg<KV, D>;
  const int l = lane_id();
  const int r = l & 15, c = l >> 4;
  const int d = 16 * m + r;
  o.x[m] = *reinterpret_cast<const u32x4*>(buf + C::KBUF + (c >> 1) * C::VBLK + d * 32 +
                                           16 * ((c & 1) ^ ((d >> 3) & 1)));
}

// S^T[32 keys x 32 columns] = K . Q^T of a pair whose K pieces are in o: s0
// holds keys 8c .. 8c + 3, s1 keys 8c + 4 .. 8c + 7 for column r of each
// N-tile. VNEXT: the pair's V tiles are read from vbuf between the MFMAs, each
// into the slots of the d-step just used, so the LDS serves them while the
// matrix core works (a wave issues in order: reads placed after the MFMAs
// would start only when the last one issues).
template <KvType KV, int D, bool VNEXT>
__device__ __forceinline__ void pf_scores(PfOps<KV, D>& o, const bf16x8 (&qb)[kPfNT][PfCfg<KV, D>::KSTEPS],
                                          f32x4 (&s0)[kPfNT], f32x4 (&s1)[kPfNT], const uint8_t* vbuf) {
  using C = PfCfg<KV, D>;
#pragma unroll
  for (int n = 0; n < kPfNT; ++n) s0[n] = s1[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < C::KSTEPS; ++j) {
    const bf16x8 k0 = __builtin_bit_cast(bf16x8, o.x[2 * j]), k1 = __builtin_bit_cast(bf16x8, o.x[2 * j + 1]);
#pragma unroll
    for (int n = 0; n < kPfNT; ++n) {
      s0[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qb[n][j], s0[n], 0, 0, 0);
      s1[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qb[n][j], s1[n], 0, 0, 0);
    }
    if constexpr (VNEXT) {
      __builtin_amdgcn_sched_barrier(0);
      pf_vread<KV, D>(vbuf, o, 2 * j);
      pf_vread<KV, D>(vbuf, o, 2 * j + 1);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// Softmax weights of one pair from its scores. MASKED: per-column key limits
// see[n] (keys of the pair the column sees). c0 / c1: softmax scale (log2
// units) times the blocks' K scales, > 0; a lane's 8 keys lie in block c / 2.
//
// The weights are exp2(logit - m) with a lazily updated running max m: only
// when a logit exceeds m by more than kSlack (so weights stay below 2^8 and fit
// fp16) is m raised and the accumulators rescaled. Each lane first checks its
// own 8 logits; the cross-lane max over the column's 4 lanes runs only when a
// lane of the wave crosses the threshold. The row sums come from a product of
// the fp16 weights with a ones operand. VMID: the first half of the pair's V
// tiles are read from vbuf once N-tile 0 is done, into registers its scores
// held, so those reads overlap N-tile 1's softmax.
template <KvType KV, int D, bool MASKED, bool VMID>
__device__ __forceinline__ void pf_softmax(const f32x4 (&s0)[kPfNT], const f32x4 (&s1)[kPfNT], float c0, float c1,
                                           const int (&see)[kPfNT], f32x4 (&acc)[PfCfg<KV, D>::MT][kPfNT],
                                           PfRow (&row)[kPfNT], f16x8 (&ph)[kPfNT], PfOps<KV, D>& o,
                                           const uint8_t* vbuf) {
  using C = PfCfg<KV, D>;
  const int l = lane_id();
  const int c = l >> 4;
  const float cs = c < 2 ? c0 : c1;
  const f16x8 ones = {1, 1, 1, 1, 1, 1, 1, 1};
#pragma unroll
  for (int n = 0; n < kPfNT; ++n) {
    float y[8];  // raw scores of keys 8c + i
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      y[i] = s0[n][i];
      y[4 + i] = s1[n][i];
    }
    if constexpr (MASKED) {
#pragma unroll
      for (int i = 0; i < 8; ++i) y[i] = 8 * c + i < see[n] ? y[i] : kNegInf;
    }
    // this lane's largest scaled logit
    const float lm =
        fmaxf(fmaxf(fmaxf(y[0], y[1]), fmaxf(y[2], y[3])), fmaxf(fmaxf(y[4], y[5]), fmaxf(y[6], y[7]))) * cs;
    if (__any(lm > row[n].m + kSlack)) {
      float mx = fmaxf(lm, __shfl_xor(lm, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(row[n].m, mx);
      const float alpha = m_new == kNegInf ? 1.f : fast_exp2(row[n].m - m_new);
      row[n].m = m_new;
      row[n].nm = m_new == kNegInf ? 0.f : -m_new;
      row[n].l *= alpha;
#pragma unroll
      for (int m = 0; m < C::MT; ++m) acc[m][n] *= alpha;
    }
    float p[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) p[i] = fast_exp2(__builtin_fmaf(y[i], cs, row[n].nm));
    u32x4 w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pk_f16(p[2 * i], p[2 * i + 1]);
    ph[n] = __builtin_bit_cast(f16x8, w);
    row[n].l = __builtin_amdgcn_mfma_f32_16x16x32_f16(ones, ph[n], row[n].l, 0, 0, 0);
    if constexpr (VMID) {
      if (n == 0) {  // the first half of the V tiles, in the registers N-tile 0's scores held
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int m = 0; m < C::MT / 2; ++m) pf_vread<KV, D>(vbuf, o, m);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
}

// O^T += V^T . P^T, V tiles VFROM .. MT - 1 read from vbuf first (the others
// are in o already). MASKED: V rows at or past `live` keys are zeroed (bitwise,
// so NaN poison in unused slots never reaches the product). KNEXT: the next
// pair's K pieces are read from kbuf between the MFMAs, each into the slot of
// the tile just used.
template <KvType KV, int D, bool MASKED, bool KNEXT, int VFROM>
__device__ __forceinline__ void pf_pv(PfOps<KV, D>& o, const f16x8 (&ph)[kPfNT], int live,
                                      f32x4 (&acc)[PfCfg<KV, D>::MT][kPfNT], const uint8_t* vbuf,
                                      const uint8_t* kbuf) {
  using C = PfCfg<KV, D>;
  static_assert(C::MT == 2 * C::KSTEPS, "one K piece per V tile");
#pragma unroll
  for (int m = VFROM; m < C::MT; ++m) pf_vread<KV, D>(vbuf, o, m);
  const int l = lane_id();
  const int c = l >> 4;
  uint32_t mk[4] = {~0u, ~0u, ~0u, ~0u};
  if constexpr (MASKED) {
#pragma unroll
    for (int h = 0; h < 4; ++h) {  // word h: keys 8c + 2h, 8c + 2h + 1
      const int k = 8 * c + 2 * h;
      mk[h] = (k < live ? 0xFFFFu : 0u) | (k + 1 < live ? 0xFFFF0000u : 0u);
    }
  }
#pragma unroll
  for (int m = 0; m < C::MT; ++m) {
    u32x4 w = o.x[m];
    if constexpr (MASKED) w = u32x4{w.x & mk[0], w.y & mk[1], w.z & mk[2], w.w & mk[3]};
    const f16x8 va = __builtin_bit_cast(f16x8, w);
#pragma unroll
    for (int n = 0; n < kPfNT; ++n) acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(va, ph[n], acc[m][n], 0, 0, 0);
    if constexpr (KNEXT) {
      __builtin_amdgcn_sched_barrier(0);
      pf_kread<KV, D>(kbuf, o, m);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

template <KvType KV, int D, bool IMG>
__global__ __launch_bounds__(kPfThreads) void prefill_kernel(PrefillArgs a) {
  using C = PfCfg<KV, D>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[4 * C::BUF];
  __shared__ int s_next[2];
  const int l = lane_id();
  const int r = l & 15, c = l >> 4;
  const int w = uni((int)(threadIdx.x >> 6));  // wave-uniform: keeps per-wave values scalar
  const uint32_t lds0 = (uint32_t)(size_t)(__attribute__((address_space(3))) uint8_t*)lds;
  const uint8_t* kimg = static_cast<const uint8_t*>(KV == KvType::FP8 ? a.k_img : a.k_cache);
  const uint8_t* vimg = static_cast<const uint8_t*>(a.v_img);
  PfLane<D> pl;
  if constexpr (IMG) pl = pf_lane<D>(w, l);
  // Unit n of queue x is item n / hq for KV head x + nq (n % hq). The grid
  // (a multiple of 8 workgroups) starts on the first gridDim / nq units of each
  // queue; each further unit is claimed with a ticket from the queue's counter
  // in the workspace header (zeroed by the plan). Unit k's claim is issued as
  // unit k starts and published in s_next[k & 1] at its first barrier; every
  // thread reads it after its last, so a slot is rewritten only after all
  // threads read it (two units later).
  const int nq = a.nq, hq = a.Hkv / nq;
  const int qsize = uni(a.hdr[kHdrItems]) * hq;  // units per queue
  const int first_claims = (int)gridDim.x / nq;
  const int xq = (int)(blockIdx.x & 7u);
  const int q = xq % nq;
  int un = (int)(blockIdx.x >> 3) * (8 / nq) + xq / nq, uq = q;  // current unit: index, queue
  int status = 0;
  for (int k = 0; un < qsize; ++k) {
    const int item = un / hq, kvh = uni(uq + nq * (un - item * hq));
    int tick = 0;
    if (threadIdx.x == 0) tick = atomicAdd(a.hdr + kHdrPfQueue + q, 1);
    const int4 it = a.items[item];
    const int b = it.x, row0 = it.y, nt = it.z, first = it.w;

    // this wave's columns: column col = 32w + 16n + r is token col / G, head col % G
    int vis[kPfNT], tokq[kPfNT];
    bf16x8 qb[kPfNT][C::KSTEPS];
    const uint32_t qflip = a.neg_scale ? 0x80008000u : 0u;  // a negative scale goes into q's sign
#pragma unroll
    for (int n = 0; n < kPfNT; ++n) {
      const int col = kPfWaveCols * w + 16 * n + r;
      const int tok = col / a.G, head = col - tok * a.G;
      const bool ok = tok < nt;
      vis[n] = first + tok + 1;  // keys the column sees
      tokq[n] = ok ? ((row0 + tok) * a.Hq + kvh * a.G + head) : -1;
      const uint16_t* qp = static_cast<const uint16_t*>(a.q) + (int64_t)(ok ? tokq[n] : 0) * D;
#pragma unroll
      for (int j = 0; j < C::KSTEPS; ++j) {
        u32x4 v = {0, 0, 0, 0};
        if (ok) v = *reinterpret_cast<const u32x4*>(qp + 32 * j + 8 * c);
        qb[n][j] = __builtin_bit_cast(bf16x8, v ^ qflip);
      }
    }
    const int tok_lo = kPfWaveCols * w / a.G;
    const int tok_hi_raw = (kPfWaveCols * w + kPfWaveCols - 1) / a.G;
    const int tok_hi = tok_hi_raw < nt - 1 ? tok_hi_raw : nt - 1;
    const bool wave_on = tok_lo < nt;
    const int pos_lo = uni(first + tok_lo);  // this wave's first and last query positions
    const int pos_hi = uni(first + tok_hi);

    const int nkeys = first + nt > 0 ? first + nt : 0;  // keys up to the tile's last position
    const int npairs = uni((nkeys + 31) / 32);
    const int nblk = uni((nkeys + 15) / 16);
    // pairs this wave computes: those with a key at or before its last position
    const int wpairs = uni(!wave_on || pos_hi < 0 ? 0 : (pos_hi / 32 + 1 < npairs ? pos_hi / 32 + 1 : npairs));
    const int32_t* row = a.block_table + uni64((int64_t)b * a.max_blocks);

    f32x4 acc[C::MT][kPfNT];
#pragma unroll
    for (int m = 0; m < C::MT; ++m)
#pragma unroll
      for (int n = 0; n < kPfNT; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
    PfRow rows[kPfNT];
#pragma unroll
    for (int n = 0; n < kPfNT; ++n) rows[n] = PfRow{kNegInf, 0.f, f32x4{0.f, 0.f, 0.f, 0.f}};

    // pair j2's weights and P . V from its scores and V tiles, on the masked
    // path where some column of the wave does not see every key of the pair, or
    // a key is past the tile; KNEXT: the next pair's K pieces are read from kbuf
    // during the P . V; VMID: half of the V tiles are read during the softmax
    // and half before the P . V (otherwise all were read during the scores)
    auto finish = [&](auto knext, auto vmid, int j2, const f32x4 (&s0)[kPfNT], const f32x4 (&s1)[kPfNT],
                      const PfMeta& m, PfOps<KV, D>& o, const uint8_t* vbuf, const uint8_t* kbuf) {
      constexpr bool KNEXT = decltype(knext)::value;
      constexpr bool VMID = decltype(vmid)::value;
      constexpr int VFROM = VMID ? C::MT / 2 : C::MT;
      const int key0 = 32 * j2;
      int see[kPfNT];
      f16x8 ph[kPfNT];
      if (key0 + 31 <= pos_lo && m.live >= 32) {
#pragma unroll
        for (int n = 0; n < kPfNT; ++n) see[n] = 32;
        pf_softmax<KV, D, false, VMID>(s0, s1, m.c0, m.c1, see, acc, rows, ph, o, vbuf);
        pf_pv<KV, D, false, KNEXT, VFROM>(o, ph, 32, acc, vbuf, kbuf);
      } else {
#pragma unroll
        for (int n = 0; n < kPfNT; ++n) see[n] = vis[n] - key0 < m.live ? vis[n] - key0 : m.live;
        pf_softmax<KV, D, true, VMID>(s0, s1, m.c0, m.c1, see, acc, rows, ph, o, vbuf);
        pf_pv<KV, D, true, KNEXT, VFROM>(o, ph, m.live, acc, vbuf, kbuf);
      }
    };

    // Two pairs per barrier: step j computes pairs j and j + 1 from LDS buffers
    // j % 4 and (j + 1) % 4 while pairs j + 2 and j + 3 travel to the other two:
    // direct loads issued at the step's start (image path), or loads into two
    // register sets that are converted and stored between the step's two pairs
    // (staging path: with their registers free, pair j + 1's V tiles fit beside
    // its softmax). The id and staging loads are unconditional (past the end
    // the last pair again, never stored), so no loaded register is merged
    // across paths: a copy of one would wait for its load at once.
    PfIds ids;
    ids.q = -1;
    ids.id = 0;
    ids.nxt = pf_id_load(row, l, nblk);  // chunk 0
    pf_ids_advance(ids, row, 0, nblk);
    PfMeta m0{1.f, 1.f, 0}, m1{1.f, 1.f, 0};
    {
      const PfPair pa = pf_pair<KV, IMG>(a, ids, 0, nblk, nkeys, kvh, status);
      const PfPair pb = pf_pair<KV, IMG>(a, ids, npairs > 1 ? 2 : 0, nblk, nkeys, kvh, status);
      if constexpr (IMG) {
        if (npairs > 0) pf_dma<KV, D>(kimg, vimg, pa.t0, pa.t1, pl, lds0);
        if (npairs > 1) pf_dma<KV, D>(kimg, vimg, pb.t0, pb.t1, pl, lds0 + C::BUF);
        pf_dma_wait();
      } else if (npairs > 0) {  // both pairs' loads before either store: one round trip
        PfStage<KV, D> sa, sb;
        pf_load<KV, D>(sa, a, pa.t0, pa.t1);
        pf_load<KV, D>(sb, a, pb.t0, pb.t1);
        pf_store<KV, D>(sa, pf_vs(pa, 0), pf_vs(pa, 1), pa.live, lds, status);
        if (npairs > 1) pf_store<KV, D>(sb, pf_vs(pb, 0), pf_vs(pb, 1), pb.live, lds + C::BUF, status);
      }
      m0 = pf_meta(pa, a.scale_log2);
      m1 = pf_meta(pb, a.scale_log2);
    }
    if (threadIdx.x == 0) {  // the next unit: 8 * index + queue, or -1 once every queue is drained
      int code = -1, m = tick + first_claims;
      if (m < qsize) code = 8 * m + q;
      for (int s = 1; s < nq && code < 0; ++s) {
        const int q2 = (q + s) % nq;
        m = atomicAdd(a.hdr + kHdrPfQueue + q2, 1) + first_claims;
        if (m < qsize) code = 8 * m + q2;
      }
      s_next[k & 1] = code;
    }
    __syncthreads();
    for (int j2 = 0; j2 < npairs; j2 += 2) {
      // blocks 2ja .. 2jb + 1 lie in one chunk of 64 (2ja is a multiple of 4, or jb = ja)
      const int ja = j2 + 2 < npairs ? j2 + 2 : npairs - 1, jb = j2 + 3 < npairs ? j2 + 3 : npairs - 1;
      pf_ids_advance(ids, row, ja >> 5, nblk);
      const PfPair pa = pf_pair<KV, IMG>(a, ids, 2 * ja, nblk, nkeys, kvh, status);
      const PfPair pb = pf_pair<KV, IMG>(a, ids, 2 * jb, nblk, nkeys, kvh, status);
      PfStage<KV, D> sa, sb;
      if constexpr (IMG) {
        if (j2 + 2 < npairs) pf_dma<KV, D>(kimg, vimg, pa.t0, pa.t1, pl, lds0 + ((j2 + 2) & 3) * C::BUF);
        if (j2 + 3 < npairs) pf_dma<KV, D>(kimg, vimg, pb.t0, pb.t1, pl, lds0 + ((j2 + 3) & 3) * C::BUF);
      } else {
        pf_load<KV, D>(sa, a, pa.t0, pa.t1);
        pf_load<KV, D>(sb, a, pb.t0, pb.t1);
      }
      PfOps<KV, D> o;
      if (j2 < wpairs) {
        // pair j2 + 1's K pieces are read during pair j2's P . V (even when
        // this wave skips pair j2 + 1: the buffer is in bounds)
        const uint8_t* ba = lds + (j2 & 3) * C::BUF;
        const uint8_t* bb = lds + ((j2 + 1) & 3) * C::BUF;
#pragma unroll
        for (int i = 0; i < C::MT; ++i) pf_kread<KV, D>(ba, o, i);
        f32x4 s0[kPfNT], s1[kPfNT];
        pf_scores<KV, D, IMG>(o, qb, s0, s1, ba);
        finish(std::true_type{}, std::integral_constant<bool, !IMG>{}, j2, s0, s1, m0, o, ba, bb);
      }
      const PfMeta m1cur = m1;
      if constexpr (!IMG) {
        if (j2 + 2 < npairs)
          pf_store<KV, D>(sa, pf_vs(pa, 0), pf_vs(pa, 1), pa.live, lds + ((j2 + 2) & 3) * C::BUF, status);
        if (j2 + 3 < npairs)
          pf_store<KV, D>(sb, pf_vs(pb, 0), pf_vs(pb, 1), pb.live, lds + ((j2 + 3) & 3) * C::BUF, status);
        m0 = pf_meta(pa, a.scale_log2);
        m1 = pf_meta(pb, a.scale_log2);
      }
      if (j2 + 1 < wpairs) {
        const uint8_t* bb = lds + ((j2 + 1) & 3) * C::BUF;
        f32x4 s0[kPfNT], s1[kPfNT];
        pf_scores<KV, D, true>(o, qb, s0, s1, bb);
        finish(std::false_type{}, std::false_type{}, j2 + 1, s0, s1, m1cur, o, bb, bb);
      }
      if constexpr (IMG) {
        pf_dma_wait();  // the next step's tiles are in LDS (and the fp8 scales in registers)
        m0 = pf_meta(pa, a.scale_log2);
        m1 = pf_meta(pb, a.scale_log2);
      }
      __syncthreads();
    }
    if (wave_on) {
#pragma unroll
      for (int n = 0; n < kPfNT; ++n) {
        const float lt = rows[n].l[0];
        if (tokq[n] < 0) continue;
        const float inv = lt > 0.f ? 1.f / lt : 0.f;
        if (a.out_bf16) {
          uint16_t* o = static_cast<uint16_t*>(a.out) + (int64_t)tokq[n] * D;
#pragma unroll
          for (int m = 0; m < C::MT; ++m)
            *reinterpret_cast<u32x2*>(o + 16 * m + 4 * c) =
                u32x2{pk_bf16(acc[m][n][0] * inv, acc[m][n][1] * inv), pk_bf16(acc[m][n][2] * inv, acc[m][n][3] * inv)};
        } else {
          float* o = static_cast<float*>(a.out) + (int64_t)tokq[n] * D;
#pragma unroll
          for (int m = 0; m < C::MT; ++m) *reinterpret_cast<f32x4*>(o + 16 * m + 4 * c) = acc[m][n] * inv;
        }
      }
    }
    const int code = s_next[k & 1];
    if (code < 0) break;
    un = code >> 3;
    uq = code & 7;
  }
  if (status) atomicOr(a.hdr + kHdrStatus, status);  // error paths only
}

template <KvType KV, int D>
void* prefill_fn(bool img) {
  return img ? reinterpret_cast<void*>(&prefill_kernel<KV, D, true>)
             : reinterpret_cast<void*>(&prefill_kernel<KV, D, false>);
}

template <KvType KV>
void* prefill_for_d(int D, bool img) {
  return D == 64 ? prefill_fn<KV, 64>(img) : prefill_fn<KV, 128>(img);
}

template <KvType KV>
void* prep_for_d(int D) {
  return D == 64 ? reinterpret_cast<void*>(&prefill_prep_kernel<KV, 64>)
                 : reinterpret_cast<void*>(&prefill_prep_kernel<KV, 128>);
}

}  // namespace

hipError_t launch_prefill(const PrefillArgs& a, KvType kv, hipStream_t s) {
  if (a.B == 0 || a.items_max == 0) return hipSuccess;
  PrefillArgs args = a;
  void* params[] = {&args};
  const bool img = a.v_img != nullptr;
  hipError_t e;
  if (img) {  // the plan and the image in one launch
    const int64_t cps = (a.max_blocks + kImgBlocks - 1) / kImgBlocks;
    void* prep = kv == KvType::FP8 ? prep_for_d<KvType::FP8>(a.D) : prep_for_d<KvType::BF16>(a.D);
    e = hipLaunchKernel(prep, dim3((unsigned)(1 + a.B * cps)), dim3(kPlanThreads), params, 0, s);
  } else {
    e = hipLaunchKernel(reinterpret_cast<void*>(&prefill_plan_kernel), dim3(1), dim3(kPlanThreads), params, 0, s);
  }
  if (e != hipSuccess) return e;
  void* fn = kv == KvType::FP8 ? prefill_for_d<KvType::FP8>(a.D, img) : prefill_for_d<KvType::BF16>(a.D, img);
  // the persistent grid: resident workgroups per CU times the CUs, a multiple
  // of 8 (the queues' start assumes it), no more than the units need
  static std::atomic<int> per_cu_memo[8];  // per kernel, queried once
  const int slot = (kv == KvType::FP8 ? 4 : 0) + (a.D == 128 ? 2 : 0) + (img ? 1 : 0);
  int per_cu = per_cu_memo[slot].load(std::memory_order_relaxed);
  if (per_cu == 0) {
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kPfThreads, 0);
    if (e != hipSuccess) return e;
    per_cu = per_cu > 0 ? per_cu : 1;
    per_cu_memo[slot].store(per_cu, std::memory_order_relaxed);
  }
  const int64_t units = (int64_t)a.items_max * a.Hkv;
  int64_t wgs = (int64_t)per_cu * a.cus;
  const int64_t need = (units + 7) / 8 * 8;
  wgs = wgs < need ? wgs : need;
  wgs = wgs / 8 * 8 > 8 ? wgs / 8 * 8 : 8;
  return hipLaunchKernel(fn, dim3((unsigned)wgs), dim3(kPfThreads), params, 0, s);
}

}  // namespace pda
