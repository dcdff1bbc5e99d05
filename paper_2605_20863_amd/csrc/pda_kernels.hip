// HIP kernels for batched paged-KV decode attention on MI355X (gfx950, CDNA4).
//
// One decode step computes, for every sequence b and query head h,
//     out[b, h] = softmax(scale * K_b q[b, h]) V_b
// over the sequence's cached tokens, read through its block table (the paged
// KV cache of the vLLM work cited in the paper's Sec. 8). Rollout decoding has
// a long-tailed length mix (Sec. 2.2), so the work split must not depend on
// how lengths are distributed:
//
// * Stream-K split. The (sequence, KV head) units are laid end to end as one
//   stream of 16-token block-heads (sequence-major, KV head minor), each unit
//   preceded by a small start cost (a segment's fixed work, in block-heads),
//   and the stream is cut into equal chunks. By default wave w of a persistent
//   grid takes chunk w, the range [w*Q, (w+1)*Q) with Q = ceil(total / waves),
//   so every wave does the same work no matter how lengths are distributed; optionally
//   the chunks are smaller and the waves take the rest from a counter in
//   arrival order. A chunk that covers a whole unit writes its normalised
//   output; otherwise it writes the unit's partial softmax state (m, l, acc)
//   to slot (unit + chunk), and the combine kernel merges a unit's partials
//   with log-sum-exp rescaling. Every wave plans from seq_lens itself (a
//   prefix sum over sequences), so one call is two launches and needs no
//   planning kernel.
//
// * Two wave kernels share that driver:
//   - MFMA (bf16 or fp8 cache, bf16 q): per pair of 16-token blocks,
//     S^T[16 tok x 16 heads] = K[16 x D] . Q^T[D x 16] on v_mfma_f32_16x16x32_bf16
//     (the GQA group's G <= 16 heads padded to 16 columns), online softmax on
//     the accumulator registers, then O^T[D x 16] += V^T[D x 32 tok] . P^T[32 x 16].
//     An entry with 17 to 32 columns (several query tokens per sequence, or a
//     shared-prefix entry serving several sequences) runs two such N-tiles on
//     the same K and V operands.
//     The score tiles' token rows are ordered so that each lane's accumulators
//     hold the weights of 8 consecutive tokens of one block, exactly what its
//     P^T operand needs: P never moves between lanes, and the lane's V^T
//     operand is one 16-byte (bf16) or 8-byte (fp8) load of one head-dim row.
//     The price is the dim-major V tile [D][16] in the cache layout. P is split
//     into two bf16 terms (hi + lo) so that rounding P costs ~2^-17, not 2^-9.
//   - Vector (any cache dtype, G <= 8): each 16-lane row owns 4 tokens; QK dot
//     products are lane-partial FMAs reduced across the row with DPP row
//     rotations; PV uses the same 4 tokens per row, so no LDS is needed.
//
// * fp8 (OCP e4m3) caches are dequantised in registers: codes convert exactly
//   to f32 / bf16; the per-(block, KV head) K scale multiplies that block's
//   logits and the V scale multiplies its softmax weights.
//
// * Masking selects, never multiplies: tokens at or past seq_len get logit
//   -inf and their V elements are replaced by 0, so NaN poison in unused cache
//   slots cannot leak (0 * NaN = NaN).

#include "pda_internal.h"

#include <stdint.h>

#include <type_traits>

namespace pda {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_inff();

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63); }
// The lane index, recomputed where it is used: values derived from it (LDS
// and output addresses of a segment's start and end) are then not hoisted
// into registers that stay live across a segment's pair loop.
__device__ __forceinline__ int lane_id_here() {
  int l = (int)(threadIdx.x & 63);
  asm volatile("" : "+v"(l));
  return l;
}
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// ------------------------------------------------------------- conversions

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __builtin_bit_cast(float, w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __builtin_bit_cast(float, w & 0xFFFF0000u); }

// Two e4m3 codes of w (bytes 0,1 or 2,3) -> two f32, exactly.
template <bool HI>
__device__ __forceinline__ f32x2 fp8_pair(uint32_t w) {
  return __builtin_amdgcn_cvt_pk_f32_fp8((int)w, HI);
}

// Four e4m3 codes -> four bf16 (two words), exactly (every e4m3 value is a
// bf16 value); one v_cvt_scalef32_pk_bf16_fp8 per pair, scale 1.
__device__ __forceinline__ u32x2 fp8x4_to_bf16x4(uint32_t w) {
  u32x2 r;
  r.x = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, false));
  r.y = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8((int)w, 1.0f, true));
  return r;
}

// f32 -> bf16 bits, round to nearest even (finite inputs; NaN stays NaN).
__device__ __forceinline__ uint32_t f32_to_bf16_bits(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (u >> 16) | 0x40u;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return u >> 16;
}

template <typename T>
__device__ __forceinline__ T ld(const void* p) {
  return *reinterpret_cast<const T*>(p);
}

// KV tiles are read exactly once per step: stream them with the nontemporal
// hint so the L2 and the last-level cache do not keep them. On MI355X plain
// 16-byte loads of random 4 KB tiles top out near 6.1 TB/s, nontemporal ones
// near 6.9 TB/s.
template <typename T>
__device__ __forceinline__ T ld_stream(const void* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const T*>(p));
}

// Inclusive prefix sum over the 64 lanes of the wave.
__device__ __forceinline__ int wave_incl_scan(int x) {
  const int l = lane_id();
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o, 64);
    if (l >= o) x += y;
  }
  return x;
}

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL,
                                                               0xF, 0xF, false));
}

// Sum over the 16 lanes of a DPP row; every lane of the row gets the total.
__device__ __forceinline__ float row_sum16(float x) {
  x += dpp<0x128>(x);  // row_ror:8
  x += dpp<0x124>(x);  // row_ror:4
  x += dpp<0x122>(x);  // row_ror:2
  x += dpp<0x121>(x);  // row_ror:1
  return x;
}

// ------------------------------------------------------------- planning

__device__ __forceinline__ int clamp_len(const DecodeArgs& a, int L) {
  return L < 0 ? 0 : (L > a.len_cap ? a.len_cap : L);
}

// One work entry: a run of blocks read through one block-table row and
// applied to up to 16 query columns (32 for a shared-prefix entry, in two
// MFMA N-tiles that share every K and V operand). In plain mode entry b is sequence b with
// its G query heads. In shared-prefix mode (GRPO-style groups of equal size
// whose members share leading blocks) entry (g, s) < n_prefix is group g's
// shared blocks applied to the heads of members s*M .. s*M + M - 1 (column r
// = member r / G, head r % G), and entry n_prefix + m is sequence m's blocks
// after its group's shared ones. Results equal plain attention over each
// sequence: the combine merges a sequence's prefix and suffix partials.
struct Entry {
  const int32_t* row;  // block ids, from the entry's first block on
  int L;               // valid tokens from the entry's first block
  int nb;              // blocks
  int qs;              // sequence of query column 0
  int ncols;           // query columns: G, or members * G
  bool may_final;      // a chunk that covers the whole entry writes the output
};

__device__ __forceinline__ Entry entry_of(const DecodeArgs& a, int v) {
  Entry e;
  if (!a.shared) {
    e.L = clamp_len(a, a.seq_lens[v]);
    e.nb = (e.L + kBlockSize - 1) / kBlockSize;
    e.row = a.block_table + (int64_t)v * a.max_blocks;
    e.qs = v;
    e.ncols = a.Qn * a.G;
    e.may_final = true;
  } else if (v < a.n_prefix) {
    const int g = v / a.nsub, s = v - g * a.nsub;
    const int S = a.sg[g];
    const int first = g * a.group_size;
    const int nm = a.group_size - s * a.M < a.M ? a.group_size - s * a.M : a.M;
    e.row = a.block_table + (int64_t)first * a.max_blocks;
    e.L = S * kBlockSize;
    e.nb = S;
    e.qs = first + s * a.M;
    e.ncols = nm * a.G;
    e.may_final = false;
  } else {
    const int m = v - a.n_prefix;
    const int S = a.sg[m / a.group_size];
    const int Lf = clamp_len(a, a.seq_lens[m]);
    const int nb = (Lf + kBlockSize - 1) / kBlockSize - S;
    e.row = a.block_table + (int64_t)m * a.max_blocks + S;
    e.L = Lf - S * kBlockSize;
    e.nb = nb > 0 ? nb : 0;
    e.qs = m;
    e.ncols = a.G;
    e.may_final = S == 0;
  }
  return e;
}

// Stream units a (entry, KV head) unit with blocks costs before its first
// block (see kUnitCostShared); every block-head is one unit.
__device__ __forceinline__ int unit_cost(const DecodeArgs& a) { return a.shared ? kUnitCostShared : kUnitCostPlain; }

// Stream-K plan, computed by every wave from seq_lens. The stream (each
// unit's start cost, then its block-heads, one stream unit each) is cut into
// chunks of Q stream units, chunk c covering [c*Q, (c+1)*Q); a chunk runs the
// blocks that start in it. In a static split Q = ceil(total / waves) and wave w runs
// chunk w only. In a dynamic split Q is smaller (chunks_max > waves chunks at
// most, none below chunk_min): wave w starts on chunk w and then takes chunks
// waves, waves + 1, ... in arrival order from a counter in the workspace
// header, so the waves the hardware serves faster read more of the stream
// (two waves sharing a SIMD are not served equally). A partial result's slot
// is (unit + chunk), not (unit + wave), so the values written and merged do
// not depend on which wave ran a chunk.
constexpr int kTileSeqs = 512;  // sequences one planning round trip covers, 8 per lane
constexpr int kLdsSeqs = 512;   // up to this many entries keep their prefix sums in LDS

struct StreamPlan {
  int64_t total;    // block-heads in the step
  int64_t chunk;    // Q
  int64_t nchunks;  // ceil(total / Q)
};

// Block counts of entries [t0, t0 + 512), lane l owning t0 + 8l .. +7 (all
// eight lengths are loaded before any is used, so the tile costs one round
// trip). incl[i] = inclusive prefix within the lane, base = the lane's
// exclusive prefix within the tile; returns the tile total. The counts are
// the ones entry_of gives.
__device__ __forceinline__ int load_tile(const DecodeArgs& a, int t0, int (&incl)[8], int& base, int& bad) {
  const int s0 = t0 + 8 * lane_id();
  int raw[8], sh[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int v = s0 + i;
    raw[i] = 0;
    sh[i] = 0;
    if (!a.shared) {
      if (v < a.E) raw[i] = a.seq_lens[v];
    } else if (v < a.n_prefix) {
      sh[i] = a.sg[v / a.nsub];
    } else if (v < a.E) {
      const int m = v - a.n_prefix;
      raw[i] = a.seq_lens[m];
      sh[i] = a.sg[m / a.group_size];
    }
  }
  int run = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const int v = s0 + i;
    int n;
    if (a.shared && v < a.n_prefix) {
      n = sh[i];
    } else {
      const int L = clamp_len(a, raw[i]);
      bad |= (L != raw[i]);
      n = (L + kBlockSize - 1) / kBlockSize - sh[i];
      n = n > 0 ? n : 0;
    }
    n = n > 0 ? n + unit_cost(a) : 0;  // stream units
    run += n;
    incl[i] = run;
  }
  const int x = wave_incl_scan(run);
  base = x - run;
  return __shfl(x, 63, 64);
}

// Wave 0 also publishes the prefix sums (cum) and Q (share) for the combine.
__device__ void plan_stream(const DecodeArgs& a, int wave, int32_t* pre, StreamPlan& p) {
  int carry = 0, bad = 0;
  for (int t0 = 0; t0 < a.E; t0 += kTileSeqs) {
    int incl[8], base;
    const int tot = load_tile(a, t0, incl, base, bad);
    const int s0 = t0 + 8 * lane_id();
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int excl = carry + base + (i ? incl[i - 1] : 0);
      if (s0 + i < a.E) {
        if (s0 + i < kLdsSeqs) pre[s0 + i] = excl;
        if (wave == 0) a.cum[s0 + i] = excl;
      }
    }
    carry += tot;
  }
  if (wave == 0 && __any(bad) && lane_id() == 0) atomicOr(a.hdr + kHdrStatus, kStatusLenClamped);
  p.total = (int64_t)uni(carry) * a.Hkv;
  int64_t q = (p.total + a.waves - 1) / a.waves;
  if (a.chunks_max > a.waves && q > a.chunk_min) {
    q = (p.total + a.chunks_max - 1) / a.chunks_max;
    if (q < a.chunk_min) q = a.chunk_min;
  }
  if (q < a.min_share) q = a.min_share;
  p.chunk = q;
  p.nchunks = (p.total + q - 1) / q;
  if (wave == 0 && lane_id() == 0) a.share[0] = (int32_t)q;
  // the prefix copy is private to this wave: order its LDS writes before its reads
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// The sequence b at which a scan for block-head pos starts (the last one whose
// first block-head is <= pos; empty sequences after it are skipped by the
// caller) and cum_b, the blocks of the sequences before it.
__device__ void locate(const DecodeArgs& a, const int32_t* pre, int64_t pos, int& b, int& cum_b) {
  const int l = lane_id_here();
  if (a.E <= kLdsSeqs) {
    // first the 64-sequence tile (its first entry), then the sequence in it
    const int nt = (a.E + 63) >> 6;
    const int head = l < nt ? pre[64 * l] : 0;
    uint64_t m = __ballot(l < nt && (int64_t)head * a.Hkv <= pos);
    const int t = __popcll(m) - 1;  // >= 0: pre[0] = 0 <= pos
    const int s = 64 * t + l;
    const int v = s < a.E ? pre[s] : 0;
    m = __ballot(s < a.E && (int64_t)v * a.Hkv <= pos);
    const int i = __popcll(m) - 1;
    b = uni(64 * t + i);
    cum_b = uni(__shfl(v, i, 64));
    return;
  }
  int carry = 0, unused = 0;
  for (int t0 = 0; t0 < a.E; t0 += kTileSeqs) {
    int incl[8], base;
    const int tot = load_tile(a, t0, incl, base, unused);
    if ((int64_t)(carry + tot) * a.Hkv > pos || t0 + kTileSeqs >= a.E) {
      const int s0 = t0 + 8 * l;
      const uint64_t m = __ballot(s0 < a.E && (int64_t)(carry + base) * a.Hkv <= pos);
      const int ln = __popcll(m) - 1;  // >= 0: lane 0 starts at carry <= pos
      int bi = 0, ci = carry + base;
#pragma unroll
      for (int i = 1; i < 8; ++i) {
        const int e = carry + base + incl[i - 1];
        if (s0 + i < a.E && (int64_t)e * a.Hkv <= pos) {
          bi = i;
          ci = e;
        }
      }
      b = uni(__shfl(s0 + bi, ln, 64));
      cum_b = uni(__shfl(ci, ln, 64));
      return;
    }
    carry += tot;
  }
  b = a.E;  // not reached for pos < total
  cum_b = carry;
}

// A segment's block ids, staged through a per-wave LDS chunk. Tile addresses
// depend on the ids, so an id read must not wait on the vector-memory counter:
// an id held in a VGPR that a conditional reload may still be filling makes
// the compiler wait for every tile load in flight at each issue. LDS reads are
// counted separately (lgkmcnt); the chunk refill, which does wait for its own
// global load, runs once per kIdChunk blocks.
constexpr int kIdChunk = 128;
constexpr int kWavesPerGroupMax = 4;  // stream-K waves per workgroup (independent)

struct BlockIds {
  const int32_t* row;
  int end;   // one past the last block of the segment
  int base;  // logical block of lds[0]
  int32_t* lds;
  __device__ void fill(int j) {
    base = j;
    for (int i = lane_id(); i < kIdChunk; i += 64) lds[i] = j + i < end ? row[j + i] : 0;
    // the chunk is private to this wave: order its LDS writes before its reads
    // (waves of one workgroup run independent ranges and never meet at a barrier)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
  __device__ int get(int j) {
    if (j >= base + kIdChunk) fill(j);
    return uni(lds[j - base]);
  }
};

// Physical block of logical block j, or block 0 with lim = rem = 0 when the
// table entry is out of range (flagged). rem = valid tokens from the block's
// first slot to the entry's end (may exceed 16), lim = min(rem, 16).
struct Blk {
  int64_t tile;  // (p * Hkv + kvh): tile index into either cache
  int p;
  int lim;
  int rem;
};

__device__ __forceinline__ Blk block_at(const DecodeArgs& a, BlockIds& ids, int j, int L, int kvh,
                                        int& status) {
  Blk r;
  int p = ids.get(j);
  int rem = L - j * kBlockSize;
  if ((unsigned)p >= (uint64_t)a.num_blocks) {
    status |= kStatusBadBlock;
    p = 0;
    rem = 0;
  }
  r.p = p;
  r.rem = rem;
  r.lim = rem > kBlockSize ? kBlockSize : rem;
  r.tile = (int64_t)p * a.Hkv + kvh;
  return r;
}

// One segment: blocks [j_lo, j_hi) of an entry under KV head kvh.
struct Seg {
  const int32_t* row;  // the entry's block ids
  int L;               // the entry's valid tokens
  int j_lo, j_hi;
  int kvh;
  int qs, ncols;       // query columns (see Entry)
  bool final;          // write the normalised output (ncols == G), else a partial
  int64_t slot;
};

// ------------------------------------------------------------- MFMA wave kernel

// K-tile loads are line-friendly: 16-byte load i of lane group c reads bytes
// [64 i + 16 c, +16) of its token row, so one instruction covers 64
// contiguous bytes of each of the 16 rows. MFMA contracts over head_dim in any
// order, so q's operand follows the same head-dim permutation (qdim below).
template <KvType KV, int D>
struct MfmaCfg {
  static constexpr int ESZ = KV == KvType::FP8 ? 1 : 2;
  static constexpr int KSTEPS = D / 32;       // 16x16x32 k-steps over head_dim
  static constexpr int NK4 = D * ESZ / 64;    // 16-byte K loads per lane per block
  static constexpr int MT = D / 16;           // 16-row output tiles of O^T
  // first head-dim index of the 8 that lane group c feeds to k-step j
  static __device__ __forceinline__ int qdim(int j, int c) {
    return KV == KvType::BF16 ? 8 * (4 * j + c) : 64 * (j >> 1) + 16 * c + 8 * (j & 1);
  }
};

// Token order of a pair of 16-token blocks (pair tokens 0-15 = block 0,
// 16-31 = block 1). The P^T operand of lane (column, c) holds the weights of
// pair tokens 8c .. 8c+7 (block c / 2), so the lane's V^T operand is 8
// consecutive tokens of one head-dim row of one block: one 16-byte (bf16) or
// 8-byte (fp8) load per M-tile. The score tiles deliver exactly those
// weights: row i of the first tile is pair token 8 (i / 4) + i % 4, row i of
// the second is that plus 4, so the accumulator lanes c hold tokens 8c .. 8c+3
// and 8c+4 .. 8c+7. Lane (r, c) therefore loads K rows of block r / 8: tokens
// 8 ((r / 4) % 2) + r % 4 and 4 more.
template <KvType KV>
using VSlice = typename std::conditional<KV == KvType::BF16, u32x4, u32x2>::type;

template <KvType KV, int D>
struct MfmaPair {
  using C = MfmaCfg<KV, D>;
  u32x4 k[2][C::NK4];  // A operands of the two score tiles
  VSlice<KV> v[C::MT]; // V^T operands: 8 tokens of block c / 2 per M-tile
  float ks[2], vs[2];
  int rem[2];  // valid tokens from each block's first slot to the entry's end
};

// K A-operand of k-step j (8 bf16: dims qdim(j, c) .. +8 of the lane's token row).
template <KvType KV, int D>
__device__ __forceinline__ bf16x8 k_operand(const u32x4 (&k)[MfmaCfg<KV, D>::NK4], int j) {
  if constexpr (KV == KvType::BF16) {
    return __builtin_bit_cast(bf16x8, k[j]);
  } else {
    const u32x4 w = k[j >> 1];
    const uint32_t w0 = (j & 1) ? w.z : w.x;
    const uint32_t w1 = (j & 1) ? w.w : w.y;
    const u32x2 a = fp8x4_to_bf16x4(w0);
    const u32x2 b = fp8x4_to_bf16x4(w1);
    u32x4 r = {a.x, a.y, b.x, b.y};
    return __builtin_bit_cast(bf16x8, r);
  }
}

template <KvType KV, int D>
__device__ __forceinline__ void mfma_issue(MfmaPair<KV, D>& bf, const DecodeArgs& a, BlockIds& ids,
                                           int j0, int j_hi, int L, int kvh, int& status) {
  using C = MfmaCfg<KV, D>;
  const int l = lane_id();
  const int r = l & 15, c = l >> 4;
  const uint8_t* kc = static_cast<const uint8_t*>(a.k_cache);
  const uint8_t* vc = static_cast<const uint8_t*>(a.v_cache);
  constexpr int64_t TILE = (int64_t)kBlockSize * D * C::ESZ;  // bytes per (block, head) tile
  const Blk b0 = block_at(a, ids, j0, L, kvh, status);
  int64_t tile1 = b0.tile;  // a missing second block reads the first's tile, all of it masked
  bf.rem[0] = b0.rem;
  bf.rem[1] = 0;
  bf.ks[1] = bf.vs[1] = 0.f;
  if (j0 + 1 < j_hi) {
    const Blk b1 = block_at(a, ids, j0 + 1, L, kvh, status);
    tile1 = b1.tile;
    bf.rem[1] = b1.rem;
    if constexpr (KV == KvType::FP8) {
      bf.ks[1] = a.kv_scales[b1.tile];
      bf.vs[1] = a.kv_scales[a.num_blocks * a.Hkv + b1.tile];
    } else {
      bf.ks[1] = bf.vs[1] = 1.f;
    }
  }
  if constexpr (KV == KvType::FP8) {
    bf.ks[0] = a.kv_scales[b0.tile];
    bf.vs[0] = a.kv_scales[a.num_blocks * a.Hkv + b0.tile];
  } else {
    bf.ks[0] = bf.vs[0] = 1.f;
  }
  const int64_t ktile = r < 8 ? b0.tile : tile1;
  const int tok = 8 * ((r >> 2) & 1) + (r & 3);
  const uint8_t* kt = kc + ktile * TILE + tok * D * C::ESZ + 16 * c;
#pragma unroll
  for (int i = 0; i < C::NK4; ++i) {
    bf.k[0][i] = ld_stream<u32x4>(kt + 64 * i);
    bf.k[1][i] = ld_stream<u32x4>(kt + 4 * D * C::ESZ + 64 * i);
  }
  const int64_t vtile = c < 2 ? b0.tile : tile1;
  const uint8_t* vt = vc + vtile * TILE + (r * kBlockSize + 8 * (c & 1)) * C::ESZ;
#pragma unroll
  for (int m = 0; m < C::MT; ++m) bf.v[m] = ld_stream<VSlice<KV>>(vt + m * 16 * kBlockSize * C::ESZ);
}

// Running-max slack (log2 units). The accumulators are rescaled only when a
// head's block maximum exceeds its reference max m_run by more than this, so
// unnormalised weights stay below 2^8 (harmless in fp32) and the rescale --
// a multiply of every accumulator -- almost never runs once a segment is under
// way. Every partial carries its own m_run, so the log-sum-exp combine is exact
// for any reference max.
constexpr float kMaxSlack = 8.f;

// One pair of 16-token blocks. MASKED handles pairs with slots that some of
// the lane's column may not see -- past the sequence end, a skipped block, or
// (several query tokens per sequence) past the column's causal end, `hide`
// tokens before the end: those tokens get logit -inf and zero V.
template <KvType KV, int D, bool MASKED, int NT>
__device__ __forceinline__ void mfma_compute(const MfmaPair<KV, D>& bf,
                                             const bf16x8 (&qb)[NT][MfmaCfg<KV, D>::KSTEPS], float scale_log2,
                                             f32x4 (&acc)[MfmaCfg<KV, D>::MT][NT], float (&m_run)[NT],
                                             float (&l_run)[NT], const int (&hide)[NT]) {
  using C = MfmaCfg<KV, D>;
  const int l = lane_id();
  const int c = l >> 4;

  // S^T = K . Q^T per N-tile of 16 columns, two 16-token tiles each: lane
  // holds pair tokens 8c .. 8c+7 of column (lane & 15), all from block c / 2
  // (first tile: 8c .. 8c+3).
  f32x4 s0[NT], s1[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) s0[n] = s1[n] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int j = 0; j < C::KSTEPS; ++j) {
    const bf16x8 k0 = k_operand<KV, D>(bf.k[0], j), k1 = k_operand<KV, D>(bf.k[1], j);
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      s0[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qb[n][j], s0[n], 0, 0, 0);
      s1[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qb[n][j], s1[n], 0, 0, 0);
    }
  }
  const bool hib = c >= 2;        // the lane's tokens are in the second block
  const int t0 = 8 * (c & 1);     // in-block slot of the lane's first token
  // scale_log2 > 0 here (a negative softmax scale enters through q's sign); a
  // zero or tiny scale leaves every weight at 1 either way
  const float cl = fmaxf(scale_log2 * (hib ? bf.ks[1] : bf.ks[0]), 1e-30f);
  // live: the lane's token slot holds a token of the entry (the V rows this
  // lane feeds to PV are these tokens, for every column); the lane's column
  // sees the token only if it is also `hide` or more slots before the end
  bool live[8];
  const int rem = hib ? bf.rem[1] : bf.rem[0];
  float y[NT][8];  // raw scores of the lane's tokens; -inf where masked
#pragma unroll
  for (int n = 0; n < NT; ++n) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      y[n][i] = s0[n][i];
      y[n][4 + i] = s1[n][i];
    }
  }
  if constexpr (MASKED) {
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      live[i] = t0 + i < rem;
#pragma unroll
      for (int n = 0; n < NT; ++n) y[n][i] = t0 + i < rem - hide[n] ? y[n][i] : kNegInf;
    }
  }
  // Lazy rescale: weights are exp2(logit - m) with the running max m raised
  // (and the partial rescaled) only when a logit exceeds m by kMaxSlack. Each
  // lane checks its own 8 logits; the max over the column's 4 lanes is taken
  // only when some lane of the wave crosses the threshold (wave-uniform).
  float lm[NT];
  bool up = false;
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    lm[n] = fmaxf(fmaxf(fmaxf(y[n][0], y[n][1]), fmaxf(y[n][2], y[n][3])),
                  fmaxf(fmaxf(y[n][4], y[n][5]), fmaxf(y[n][6], y[n][7]))) * cl;
    up |= lm[n] > m_run[n] + kMaxSlack;  // -inf + slack = -inf starts a segment
  }
  if (__any(up)) {
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      float mx = fmaxf(lm[n], __shfl_xor(lm[n], 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float m_new = fmaxf(m_run[n], mx);
      const float alpha = m_new == kNegInf ? 1.f : fast_exp2(m_run[n] - m_new);
      m_run[n] = m_new;
      l_run[n] *= alpha;
#pragma unroll
      for (int m = 0; m < C::MT; ++m) acc[m][n] *= alpha;
    }
  }

  // P^T operands in two bf16 terms: p = hi + lo + O(2^-17 p).
  bf16x8 phi[NT], plo[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const float nm = m_run[n] == kNegInf ? 0.f : -m_run[n];
    float p[8];
    float psum = 0.f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      p[i] = fast_exp2(__builtin_fmaf(y[n][i], cl, nm));
      psum += p[i];
    }
    l_run[n] += psum;
    if constexpr (KV == KvType::FP8) {
      const float vsl = hib ? bf.vs[1] : bf.vs[0];
#pragma unroll
      for (int i = 0; i < 8; ++i) p[i] *= vsl;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const __bf16 h = (__bf16)p[i];
      phi[n][i] = h;
      plo[n][i] = (__bf16)(p[i] - (float)h);
    }
  }
  uint32_t mk[4] = {~0u, ~0u, ~0u, ~0u};
  if constexpr (MASKED) {
    // select, so NaN poison in dead slots cannot leak through 0 * NaN
#pragma unroll
    for (int h = 0; h < 4; ++h) mk[h] = (live[2 * h] ? 0xFFFFu : 0u) | (live[2 * h + 1] ? 0xFFFF0000u : 0u);
  }
  // O^T += V^T . P^T: one V operand per M-tile serves every N-tile
#pragma unroll
  for (int m = 0; m < C::MT; ++m) {
    u32x4 w;
    if constexpr (KV == KvType::BF16) {
      w = bf.v[m];
    } else {
      const u32x2 a = fp8x4_to_bf16x4(bf.v[m].x);
      const u32x2 b = fp8x4_to_bf16x4(bf.v[m].y);
      w = u32x4{a.x, a.y, b.x, b.y};
    }
    if constexpr (MASKED) w = u32x4{w.x & mk[0], w.y & mk[1], w.z & mk[2], w.w & mk[3]};
    const bf16x8 va = __builtin_bit_cast(bf16x8, w);
#pragma unroll
    for (int n = 0; n < NT; ++n) {
      acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, phi[n], acc[m][n], 0, 0, 0);
      acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, plo[n], acc[m][n], 0, 0, 0);
    }
  }
}

// `full`: rem at which every column sees all 16 tokens of a block (16 plus
// the largest `hide`, wave-uniform).
template <KvType KV, int D, int NT>
__device__ __forceinline__ void mfma_step(const MfmaPair<KV, D>& bf, const bf16x8 (&qb)[NT][MfmaCfg<KV, D>::KSTEPS],
                                          float scale_log2, f32x4 (&acc)[MfmaCfg<KV, D>::MT][NT],
                                          float (&m_run)[NT], float (&l_run)[NT], int full, const int (&hide)[NT]) {
  if (bf.rem[0] >= full && bf.rem[1] >= full)
    mfma_compute<KV, D, false, NT>(bf, qb, scale_log2, acc, m_run, l_run, hide);
  else
    mfma_compute<KV, D, true, NT>(bf, qb, scale_log2, acc, m_run, l_run, hide);
}

// NT N-tiles of 16 query columns: 1 for entries of up to 16 columns, 2 for
// up to 32 (the prefix entries of shared-prefix mode, with several members'
// heads per shared block, or several query tokens per sequence). DEPTH pairs
// in flight: 3 or 2 (the two-tile body has the registers for 2; the wide
// kernel gives every segment the same depth, so the waves that carry two-tile
// entries keep as many bytes in flight as the others and take an even share
// of the bandwidth).
// claim: this is the last segment of a chunk of a dynamic split; the claim for
// the wave's next chunk (an atomic on the workspace counter, into `ticket` of
// lane 0) is issued right after the segment's last tile loads.
template <KvType KV, int D, int NT, int DEPTH>
__device__ void mfma_segment(const DecodeArgs& a, const Seg& sg, int& status, int32_t* id_lds, bool claim,
                             int& ticket) {
  using C = MfmaCfg<KV, D>;
  const int l = lane_id();
  const int r = l & 15, c = l >> 4;
  const int kvh = sg.kvh, L = sg.L, j_lo = sg.j_lo, j_hi = sg.j_hi;

  // Q^T B-operand of N-tile n: column col = 16n + r = (mem, head) with
  // mem = col / G the member (shared-prefix entries) or the query token
  // (several per sequence), dims qdim(j, c) .. +8 for k-step j. q rows are
  // [sequence, query token, head].
  int qo_row[NT];  // < 2^31: the host bounds num_seqs * q_tokens * num_q_heads
  int hide[NT];
  bool on[NT];
  const int full = kBlockSize + a.Qn - 1;
  bf16x8 qb[NT][C::KSTEPS];
  const uint32_t qflip = a.neg_scale ? 0x80008000u : 0u;  // a negative scale goes into q's sign
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    const int col = 16 * n + r;
    const int mem = col / a.G, head = col - mem * a.G;
    on[n] = col < sg.ncols;
    qo_row[n] = (sg.qs * a.Qn + mem) * a.Hq + kvh * a.G + head;
    // query token mem of Qn sits Qn - 1 - mem tokens before the sequence end
    hide[n] = a.Qn > 1 && mem < a.Qn ? a.Qn - 1 - mem : 0;
    const uint16_t* qrow = static_cast<const uint16_t*>(a.q) + (int64_t)(on[n] ? qo_row[n] : 0) * D;
#pragma unroll
    for (int j = 0; j < C::KSTEPS; ++j) {
      u32x4 w = {0, 0, 0, 0};
      if (on[n]) w = ld<u32x4>(qrow + C::qdim(j, c));
      qb[n][j] = __builtin_bit_cast(bf16x8, w ^ qflip);
    }
  }

  BlockIds ids{sg.row, j_hi, 0, id_lds};
  ids.fill(j_lo);

  f32x4 acc[C::MT][NT];
#pragma unroll
  for (int m = 0; m < C::MT; ++m)
#pragma unroll
    for (int n = 0; n < NT; ++n) acc[m][n] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m_run[NT], l_run[NT];
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    m_run[n] = kNegInf;
    l_run[n] = 0.f;
  }

  const int npairs = (j_hi - j_lo + 1) >> 1;
  auto step = [&](const MfmaPair<KV, D>& bf) {
    mfma_step<KV, D, NT>(bf, qb, a.mfma_scale_log2, acc, m_run, l_run, full, hide);
  };
  auto issue = [&](MfmaPair<KV, D>& bf, int p) { mfma_issue<KV, D>(bf, a, ids, j_lo + 2 * p, j_hi, L, kvh, status); };
  // The claim follows the last pair's loads: vector-memory operations complete
  // in issue order for s_waitcnt, so a claim issued earlier would hold up every
  // tile wait after it for the atomic's round trip.
  auto claim_next = [&]() {
    if (claim && l == 0) ticket = atomicAdd(a.hdr + kHdrNext, 1);
  };
  static_assert(DEPTH == 2 || DEPTH == 3, "pairs in flight");
  if constexpr (DEPTH == 3) {
    // three pairs in flight (one bf16 wave per SIMD leaves the registers for it)
    MfmaPair<KV, D> b0, b1, b2;
    if (npairs > 0) issue(b0, 0);
    if (npairs > 1) issue(b1, 1);
    if (npairs > 2) issue(b2, 2);
    int i = 0;
    for (; i + 5 < npairs; i += 3) {
      step(b0);
      issue(b0, i + 3);
      step(b1);
      issue(b1, i + 4);
      step(b2);
      issue(b2, i + 5);
    }
    // at most five pairs left: i, i+1, i+2 in flight in b0, b1, b2
    if (i < npairs) {
      step(b0);
      if (i + 3 < npairs) issue(b0, i + 3);
    }
    if (i + 1 < npairs) {
      step(b1);
      if (i + 4 < npairs) issue(b1, i + 4);
    }
    claim_next();  // every pair is issued
    if (i + 2 < npairs) step(b2);
    if (i + 3 < npairs) step(b0);
    if (i + 4 < npairs) step(b1);
  } else {
    MfmaPair<KV, D> b0, b1;
    if (npairs > 0) issue(b0, 0);
    if (npairs > 1) issue(b1, 1);
    int i = 0;
    for (; i + 3 < npairs; i += 2) {
      step(b0);
      issue(b0, i + 2);
      step(b1);
      issue(b1, i + 3);
    }
    if (i < npairs) {
      step(b0);
      if (i + 2 < npairs) issue(b0, i + 2);
    }
    claim_next();  // every pair is issued
    if (i + 1 < npairs) step(b1);
    if (i + 2 < npairs) step(b0);
  }

  // the output section takes the lane index afresh: addresses derived from it
  // here are then formed here, not kept in registers across the pair loop
  const int lo = lane_id_here();
  const int ro = lo & 15, co = lo >> 4;
#pragma unroll
  for (int n = 0; n < NT; ++n) {
    // Lanes c = 0..3 hold disjoint token subsets of column r: total the denominator.
    float lt = l_run[n];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    if (!on[n]) continue;
    if (sg.final) {  // plain entry: the column is query token mem, head `head` of sequence qs
      const float inv = lt > 0.f ? 1.f / lt : 0.f;
      // the row index stays live across the pair loop, the address is formed
      // only here (an address formed at the start would hold two more registers)
      int qrow_end = qo_row[n];
      asm volatile("" : "+v"(qrow_end));
      const int64_t orow = (int64_t)qrow_end * D;
      if (a.out_bf16) {
        uint16_t* o = static_cast<uint16_t*>(a.out) + orow;
#pragma unroll
        for (int m = 0; m < C::MT; ++m) {
          u32x2 w;
          w.x = f32_to_bf16_bits(acc[m][n][0] * inv) | (f32_to_bf16_bits(acc[m][n][1] * inv) << 16);
          w.y = f32_to_bf16_bits(acc[m][n][2] * inv) | (f32_to_bf16_bits(acc[m][n][3] * inv) << 16);
          *reinterpret_cast<u32x2*>(o + 16 * m + 4 * co) = w;
        }
      } else {
        float* o = static_cast<float*>(a.out) + orow;
#pragma unroll
        for (int m = 0; m < C::MT; ++m) *reinterpret_cast<f32x4*>(o + 16 * m + 4 * co) = acc[m][n] * inv;
      }
    } else {
      const int64_t prow = sg.slot * a.Gp + 16 * n + ro;
      float* arow = a.ws_acc + prow * D;
#pragma unroll
      for (int m = 0; m < C::MT; ++m) *reinterpret_cast<f32x4*>(arow + 16 * m + 4 * co) = acc[m][n];
      if (co == 0) {
        a.ws_m[prow] = m_run[n];
        a.ws_l[prow] = lt;
      }
    }
  }
}

// ------------------------------------------------------------- vector wave kernel

template <KvType KV, int D>
struct VecCfg {
  static constexpr int ESZ = KV == KvType::F32 ? 4 : (KV == KvType::BF16 ? 2 : 1);
  static constexpr int ED = D / 16;          // dims per lane (K side) / dim rows per lane (V side)
  static constexpr int KW = ED * ESZ / 4;    // words per lane per token (K)
  static constexpr int VW = ESZ;             // words per lane per dim row (4 tokens)
};

template <KvType KV, int D>
struct VecBlock {
  using C = VecCfg<KV, D>;
  uint32_t k[4][C::KW];
  uint32_t v[C::ED][C::VW];
  float ks, vs;
  int lim;
};

template <int N>
__device__ __forceinline__ void ld_words(uint32_t (&dst)[N], const uint8_t* p) {
  if constexpr (N % 4 == 0) {
#pragma unroll
    for (int i = 0; i < N; i += 4) {
      const u32x4 w = ld_stream<u32x4>(p + 4 * i);
      dst[i] = w.x; dst[i + 1] = w.y; dst[i + 2] = w.z; dst[i + 3] = w.w;
    }
  } else if constexpr (N == 2) {
    const u32x2 w = ld_stream<u32x2>(p);
    dst[0] = w.x; dst[1] = w.y;
  } else {
    dst[0] = ld_stream<uint32_t>(p);
  }
}

// Decode N stored elements (packed in words) to f32.
template <KvType KV, int N, int W>
__device__ __forceinline__ void decode_elems(float (&f)[N], const uint32_t (&w)[W]) {
  if constexpr (KV == KvType::F32) {
#pragma unroll
    for (int i = 0; i < N; ++i) f[i] = __builtin_bit_cast(float, w[i]);
  } else if constexpr (KV == KvType::BF16) {
#pragma unroll
    for (int i = 0; i < N / 2; ++i) {
      f[2 * i] = bf16_lo(w[i]);
      f[2 * i + 1] = bf16_hi(w[i]);
    }
  } else {
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
      const f32x2 lo = fp8_pair<false>(w[i]);
      const f32x2 hi = fp8_pair<true>(w[i]);
      f[4 * i] = lo.x; f[4 * i + 1] = lo.y; f[4 * i + 2] = hi.x; f[4 * i + 3] = hi.y;
    }
  }
}

template <KvType KV, int D>
__device__ __forceinline__ void vec_issue(VecBlock<KV, D>& bk, const DecodeArgs& a, BlockIds& ids, int j,
                                          int L, int kvh, int& status) {
  using C = VecCfg<KV, D>;
  const int l = lane_id();
  const int r4 = l >> 4, c16 = l & 15;
  const Blk blk = block_at(a, ids, j, L, kvh, status);
  bk.lim = blk.lim;
  constexpr int64_t TILE = (int64_t)kBlockSize * D * C::ESZ;
  const uint8_t* kt = static_cast<const uint8_t*>(a.k_cache) + blk.tile * TILE;
  const uint8_t* vt = static_cast<const uint8_t*>(a.v_cache) + blk.tile * TILE;
#pragma unroll
  for (int jj = 0; jj < 4; ++jj)
    ld_words<C::KW>(bk.k[jj], kt + ((4 * r4 + jj) * D + c16 * C::ED) * C::ESZ);
#pragma unroll
  for (int e = 0; e < C::ED; ++e)
    ld_words<C::VW>(bk.v[e], vt + ((c16 + 16 * e) * kBlockSize + 4 * r4) * C::ESZ);
  if constexpr (KV == KvType::FP8) {
    bk.ks = a.kv_scales[blk.tile];
    bk.vs = a.kv_scales[a.num_blocks * a.Hkv + blk.tile];
  } else {
    bk.ks = 1.f;
    bk.vs = 1.f;
  }
}

template <KvType KV, int D, int GV, bool MASKED>
__device__ __forceinline__ void vec_compute(const VecBlock<KV, D>& bk, const float (&qf)[GV][VecCfg<KV, D>::ED],
                                            float scale_log2, float (&acc)[GV][VecCfg<KV, D>::ED],
                                            float (&m_run)[GV], float (&l_run)[GV]) {
  using C = VecCfg<KV, D>;
  const int r4 = lane_id() >> 4;
  const float coef = scale_log2 * bk.ks;
  bool valid[4];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) valid[jj] = !MASKED || 4 * r4 + jj < bk.lim;
  // logits of this row's 4 tokens for every head: lane-partial dot products
  // over D/16 dims, reduced across the 16-lane row
  float x[4][GV];
#pragma unroll
  for (int jj = 0; jj < 4; ++jj) {
    float kf[C::ED];
    decode_elems<KV, C::ED, C::KW>(kf, bk.k[jj]);
#pragma unroll
    for (int h = 0; h < GV; ++h) {
      float part = 0.f;
#pragma unroll
      for (int e = 0; e < C::ED; ++e) part = fmaf(qf[h][e], kf[e], part);
      const float sx = row_sum16(part) * coef;
      x[jj][h] = valid[jj] ? sx : kNegInf;
    }
  }
  // V rows (c16 + 16e) x this row's 4 tokens; dead slots selected to 0
  float vf[C::ED][4];
#pragma unroll
  for (int e = 0; e < C::ED; ++e) {
    float t4[4];
    decode_elems<KV, 4, C::VW>(t4, bk.v[e]);
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) vf[e][jj] = valid[jj] ? t4[jj] : 0.f;
  }
  float mx[GV];
  bool grow = false;
#pragma unroll
  for (int h = 0; h < GV; ++h) {
    float m = fmaxf(fmaxf(x[0][h], x[1][h]), fmaxf(x[2][h], x[3][h]));
    m = fmaxf(m, __shfl_xor(m, 16, 64));
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    mx[h] = m;
    grow |= m > m_run[h] + kMaxSlack;
  }
  if (__any(grow)) {  // wave-uniform lazy rescale, as in the MFMA kernel
#pragma unroll
    for (int h = 0; h < GV; ++h) {
      const float m_new = fmaxf(m_run[h], mx[h]);
      const float alpha = m_new == kNegInf ? 1.f : fast_exp2(m_run[h] - m_new);
      m_run[h] = m_new;
      l_run[h] *= alpha;
#pragma unroll
      for (int e = 0; e < C::ED; ++e) acc[h][e] *= alpha;
    }
  }
#pragma unroll
  for (int h = 0; h < GV; ++h) {
    const float m_ref = m_run[h] == kNegInf ? 0.f : m_run[h];
    float p[4];
    float psum = 0.f;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      p[jj] = fast_exp2(x[jj][h] - m_ref);
      psum += p[jj];
    }
    l_run[h] += psum;
    if constexpr (KV == KvType::FP8) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) p[jj] *= bk.vs;
    }
#pragma unroll
    for (int e = 0; e < C::ED; ++e) {
      float t = acc[h][e];
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) t = fmaf(p[jj], vf[e][jj], t);
      acc[h][e] = t;
    }
  }
}

template <KvType KV, int D, int GV>
__device__ __forceinline__ void vec_step(const VecBlock<KV, D>& bk, const float (&qf)[GV][VecCfg<KV, D>::ED],
                                         float scale_log2, float (&acc)[GV][VecCfg<KV, D>::ED],
                                         float (&m_run)[GV], float (&l_run)[GV]) {
  if (bk.lim == kBlockSize)
    vec_compute<KV, D, GV, false>(bk, qf, scale_log2, acc, m_run, l_run);
  else
    vec_compute<KV, D, GV, true>(bk, qf, scale_log2, acc, m_run, l_run);
}

// Plain mode only (the host sends shared-prefix calls to the MFMA kernel).
template <KvType KV, int D, int GV>
__device__ void vec_segment(const DecodeArgs& a, const Seg& sg, int& status, int32_t* id_lds, bool claim,
                            int& ticket) {
  using C = VecCfg<KV, D>;
  const int l = lane_id();
  const int r4 = l >> 4, c16 = l & 15;
  const int b = sg.qs, kvh = sg.kvh, L = sg.L, j_lo = sg.j_lo, j_hi = sg.j_hi;
  const bool final = sg.final;
  const int64_t slot = sg.slot;

  float qf[GV][C::ED];
#pragma unroll
  for (int h = 0; h < GV; ++h) {
    const int64_t row = ((int64_t)b * a.Hq + kvh * a.G + h) * D + c16 * C::ED;
#pragma unroll
    for (int e = 0; e < C::ED; ++e) {
      float v = 0.f;
      if (h < a.G) {
        if constexpr (KV == KvType::F32) {
          v = static_cast<const float*>(a.q)[row + e];
        } else {
          v = __builtin_bit_cast(float, (uint32_t) static_cast<const uint16_t*>(a.q)[row + e] << 16);
        }
      }
      qf[h][e] = v;
    }
  }

  BlockIds ids{sg.row, j_hi, 0, id_lds};
  ids.fill(j_lo);

  float acc[GV][C::ED];
  float m_run[GV], l_run[GV];
#pragma unroll
  for (int h = 0; h < GV; ++h) {
    m_run[h] = kNegInf;
    l_run[h] = 0.f;
#pragma unroll
    for (int e = 0; e < C::ED; ++e) acc[h][e] = 0.f;
  }

  const int n = j_hi - j_lo;
  VecBlock<KV, D> b0, b1;
  auto issue = [&](VecBlock<KV, D>& bk, int i) { vec_issue<KV, D>(bk, a, ids, j_lo + i, L, kvh, status); };
  if (n > 0) issue(b0, 0);
  if (n > 1) issue(b1, 1);
  int i = 0;
  for (; i + 3 < n; i += 2) {
    vec_step<KV, D, GV>(b0, qf, a.scale_log2, acc, m_run, l_run);
    issue(b0, i + 2);
    vec_step<KV, D, GV>(b1, qf, a.scale_log2, acc, m_run, l_run);
    issue(b1, i + 3);
  }
  if (i < n) {
    vec_step<KV, D, GV>(b0, qf, a.scale_log2, acc, m_run, l_run);
    if (i + 2 < n) issue(b0, i + 2);
  }
  // as in the MFMA body, the claim follows the last block's loads
  if (claim && l == 0) ticket = atomicAdd(a.hdr + kHdrNext, 1);
  if (i + 1 < n) vec_step<KV, D, GV>(b1, qf, a.scale_log2, acc, m_run, l_run);
  if (i + 2 < n) vec_step<KV, D, GV>(b0, qf, a.scale_log2, acc, m_run, l_run);

  // Each 16-lane row holds its own 4-token subsets: total over the 4 rows.
#pragma unroll
  for (int h = 0; h < GV; ++h) {
    l_run[h] += __shfl_xor(l_run[h], 16, 64);
    l_run[h] += __shfl_xor(l_run[h], 32, 64);
#pragma unroll
    for (int e = 0; e < C::ED; ++e) {
      acc[h][e] += __shfl_xor(acc[h][e], 16, 64);
      acc[h][e] += __shfl_xor(acc[h][e], 32, 64);
    }
  }
  if (r4 != 0) return;
#pragma unroll
  for (int h = 0; h < GV; ++h) {
    if (h >= a.G) break;
    const int hq = kvh * a.G + h;
    if (final) {
      const float inv = l_run[h] > 0.f ? 1.f / l_run[h] : 0.f;
      const int64_t orow = ((int64_t)b * a.Hq + hq) * D;
#pragma unroll
      for (int e = 0; e < C::ED; ++e) {
        const float o = acc[h][e] * inv;
        if (a.out_bf16) {
          static_cast<uint16_t*>(a.out)[orow + c16 + 16 * e] = (uint16_t)f32_to_bf16_bits(o);
        } else {
          static_cast<float*>(a.out)[orow + c16 + 16 * e] = o;
        }
      }
    } else {
      float* arow = a.ws_acc + (slot * a.Gp + h) * D;
#pragma unroll
      for (int e = 0; e < C::ED; ++e) arow[c16 + 16 * e] = acc[h][e];
      if (c16 == 0) {
        a.ws_m[slot * a.Gp + h] = m_run[h];
        a.ws_l[slot * a.Gp + h] = l_run[h];
      }
    }
  }
}

// ------------------------------------------------------------- persistent driver

template <Variant V, KvType KV, int D, int GV>
__device__ __forceinline__ void decode_body(const DecodeArgs& a) {
  __shared__ int32_t id_lds_all[kWavesPerGroupMax][kIdChunk];
  __shared__ int32_t pre_all[kWavesPerGroupMax][kLdsSeqs];
  const int wave_in_group = uni(threadIdx.x >> 6);  // wave-uniform: the LDS bases stay in scalar registers
  int32_t* id_lds = id_lds_all[wave_in_group];
  int32_t* pre = pre_all[wave_in_group];
  const int wave = blockIdx.x * (blockDim.x >> 6) + wave_in_group;
  StreamPlan plan;
  plan_stream(a, wave, pre, plan);
  const bool dynamic = plan.nchunks > a.waves;
  int status = 0;
  for (int64_t c = wave; c < plan.nchunks;) {
    // A dynamic split claims the wave's next chunk from the counter near the end
    // of this one: after the tile loads of its last segment, so the claims come
    // in the order waves finish and the round trip overlaps the last pairs'
    // work. A chunk whose last segment is not known in advance (the chunk ends
    // in a unit's start cost), or that holds no blocks, claims after its loop.
    int ticket = 0;
    bool claimed = !dynamic;
    int64_t pos = c * plan.chunk;
    const int64_t end = pos + plan.chunk < plan.total ? pos + plan.chunk : plan.total;
    int v, cum_v;
    locate(a, pre, pos, v, cum_v);
    while (pos < end && v < a.E) {
      const Entry e = entry_of(a, v);
      const int nb = e.nb;
      // the entry's units in stream units: KV head kvh's blocks occupy
      // [base + kvh * nbw, base + (kvh + 1) * nbw), block j starting at j * wt
      // (offsets within an entry fit in 32 bits: the host bounds entries *
      // blocks * KV heads * weight by INT32_MAX)
      const int f = nb > 0 ? unit_cost(a) : 0;  // block j starts at f + j
      const int nbw = f + nb;
      const int64_t base = (int64_t)cum_v * a.Hkv;
      if (pos >= base + (int64_t)nbw * a.Hkv) {
        cum_v += nbw;
        ++v;
        continue;
      }
      const int rel = (int)(pos - base);
      const int kvh = rel / nbw;
      const int r0 = rel - kvh * nbw;  // pos within the unit
      const int64_t u0 = pos - r0;     // the unit's first stream unit
      const int r_end = end - u0 < nbw ? (int)(end - u0) : nbw;
      // this chunk's blocks: those that start in [pos, end)
      const int j_lo = r0 > f ? r0 - f : 0;
      const int j_hi = r_end > f ? r_end - f : 0;
      // on to the start of block j_hi, or past the unit
      const int64_t next = u0 + (j_hi < nb ? f + j_hi : nbw);
      if (j_lo < j_hi) {
        const Seg sg{e.row, e.L, j_lo, j_hi, kvh, e.qs, e.ncols, e.may_final && j_lo == 0 && j_hi == nb,
                     (int64_t)v * a.Hkv + kvh + c};
        // the chunk's last segment: it reaches the chunk's end, or no entry follows
        const bool claim = !claimed && (next >= end || (j_hi == nb && kvh + 1 == a.Hkv && v + 1 >= a.E));
        claimed |= claim;
        if constexpr (V == Variant::Mfma && GV == kWideColumns) {
          // wide kernel: shared-prefix prefix entries, or several query tokens
          // per sequence, carry up to 32 columns
          if (sg.ncols > 16) mfma_segment<KV, D, 2, 2>(a, sg, status, id_lds, claim, ticket);
          else mfma_segment<KV, D, 1, 2>(a, sg, status, id_lds, claim, ticket);
        } else if constexpr (V == Variant::Mfma) {
          mfma_segment<KV, D, 1, KV == KvType::BF16 ? 3 : 2>(a, sg, status, id_lds, claim, ticket);
        } else {
          vec_segment<KV, D, GV>(a, sg, status, id_lds, claim, ticket);
        }
      }
      pos = next;
    }
    if (!claimed && lane_id() == 0) ticket = atomicAdd(a.hdr + kHdrNext, 1);
    c = dynamic ? (int64_t)a.waves + uni(ticket) : plan.nchunks;
  }
  if (__any(status) && lane_id() == 0) atomicOr(a.hdr + kHdrStatus, status);
}

// The read-only inputs also arrive as __restrict__ kernel parameters: with
// them marked noalias the compiler may read block ids and fp8 scales through
// the scalar cache (the kernel's own stores to the workspace cannot clobber
// them), which keeps id lookups off the vector-memory counter.
__device__ __forceinline__ DecodeArgs with_inputs(DecodeArgs a, const void* __restrict__ q,
                                                  const void* __restrict__ kc, const void* __restrict__ vc,
                                                  const int32_t* __restrict__ bt,
                                                  const int32_t* __restrict__ lens,
                                                  const float* __restrict__ scales) {
  a.q = q;
  a.k_cache = kc;
  a.v_cache = vc;
  a.block_table = bt;
  a.seq_lens = lens;
  a.kv_scales = scales;
  return a;
}

template <Variant V, KvType KV, int D, int GV>
__global__ __launch_bounds__(256) void decode_kernel(
    DecodeArgs a, const void* __restrict__ q, const void* __restrict__ kc, const void* __restrict__ vc,
    const int32_t* __restrict__ bt, const int32_t* __restrict__ lens, const float* __restrict__ scales) {
  decode_body<V, KV, D, GV>(with_inputs(a, q, kc, vc, bt, lens, scales));
}

// fp8 MFMA waves are held to two per SIMD (<= 256 VGPR + AGPR): the fp8 body
// spends more VALU time per byte, and a second wave per SIMD covers it.
template <Variant V, KvType KV, int D, int GV>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2, 2))) void decode_kernel_occ2(
    DecodeArgs a, const void* __restrict__ q, const void* __restrict__ kc, const void* __restrict__ vc,
    const int32_t* __restrict__ bt, const int32_t* __restrict__ lens, const float* __restrict__ scales) {
  decode_body<V, KV, D, GV>(with_inputs(a, q, kc, vc, bt, lens, scales));
}

template <Variant V, KvType KV, int D, int GV>
__global__ __launch_bounds__(256) void decode_kernel_vec(
    DecodeArgs a, const void* __restrict__ q, const void* __restrict__ kc, const void* __restrict__ vc,
    const int32_t* __restrict__ bt, const int32_t* __restrict__ lens, const float* __restrict__ scales) {
  decode_body<V, KV, D, GV>(with_inputs(a, q, kc, vc, bt, lens, scales));
}

// ------------------------------------------------------------- LSE combine

constexpr int kCombineThreads = 256;
constexpr int kCombineChunk = 8;  // segments whose loads are in flight together

// One workgroup per (sequence, KV head): merges the partial softmax states
// (m_w, l_w, acc_w) of the chunks w that computed parts of the sequence's
// attention for that head,
//     out = sum_w 2^(m_w - M) acc_w / sum_w 2^(m_w - M) l_w,   M = max_w m_w,
// and writes zeros for empty sequences. The partials come from up to two
// entries: the sequence's own (its suffix in shared-prefix mode) and, in
// shared-prefix mode, its group's prefix entry, whose columns
// col0 .. col0 + G - 1 are this sequence's heads. The kernel is latency-bound
// (a few KB per sequence and head), so it is organised around round trips:
// one for the entries' chunk ranges, then one per group of 8 chunks in which
// every thread loads the (m, l) of its head and its accumulator elements
// together and folds them in with a running maximum.
template <bool OUT_BF16, int D>
__global__ __launch_bounds__(kCombineThreads) void combine_kernel(DecodeArgs a) {
  // the decode kernel has finished with the chunk counter: rearm it for the next call
  if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0) a.hdr[kHdrNext] = 0;
  const int u = blockIdx.x;
  const int b = u / a.Hkv;
  const int kvh = u - b * a.Hkv;
  const int G = a.G;
  const int tid = threadIdx.x;
  // this sequence's columns for the KV head: G heads times its query tokens;
  // workgroup y takes columns 16y .. 16y + 15 of them
  const int ncol = a.Qn * G;
  const int cbase = 16 * (int)blockIdx.y;
  // Every value the segment ranges need, loaded at once (one round trip):
  // the length, the prefix sums of the sequence's entries and Q, and in
  // shared-prefix mode the group's shared blocks. All indices are in range in
  // either mode (in plain mode g = 0 and the shared-block read goes to cum[0]).
  const int g = a.shared ? b / a.group_size : 0;
  const int mi = b - g * a.group_size;  // member index in the group
  const int sub = a.shared ? mi / a.M : 0;
  const int v_own = a.shared ? a.n_prefix + b : b;
  const int v_pre = g * a.nsub + sub;
  const int32_t* sgp = a.shared ? a.sg : a.cum;
  const int raw = a.seq_lens[b];
  const int cum_own = a.cum[v_own];
  const int cum_pre = a.cum[a.shared ? v_pre : 0];
  const int S = sgp[g];
  const int share32 = a.share[0];
  // keep Q's load beside the others (the compiler would sink it into the
  // branch that uses it, one more round trip)
  asm volatile("" ::"v"(share32));
  const int64_t share = share32;

  int64_t slot0[2];
  int nseg[2], col0[2];
  int parts = 0;
  // the sequence's own entry (its suffix after the shared blocks in shared-prefix mode)
  const int Lf = clamp_len(a, raw);
  const int S_own = a.shared ? S : 0;
  const int nb_raw = (Lf + kBlockSize - 1) / kBlockSize - S_own;
  const int own_nb = nb_raw > 0 ? nb_raw : 0;
  const bool own_may_final = S_own == 0;
  // a unit's segments: the chunks from the one holding its first block to
  // the one holding its last (its start cost, before the first block, may
  // end a chunk that holds none of its blocks)
  if (own_nb > 0) {
    const int f = unit_cost(a);
    const int64_t start = (int64_t)cum_own * a.Hkv + (int64_t)kvh * (f + own_nb) + f;
    const int64_t w0 = start / share;
    nseg[parts] = (int)((start + own_nb - 1) / share - w0) + 1;
    slot0[parts] = (int64_t)v_own * a.Hkv + kvh + w0;
    col0[parts] = 0;
    ++parts;
  }
  if (a.shared && S > 0) {  // the group's prefix entry: columns of member i
    const int f = unit_cost(a);
    const int64_t start = (int64_t)cum_pre * a.Hkv + (int64_t)kvh * (f + S) + f;
    const int64_t w0 = start / share;
    nseg[parts] = (int)((start + S - 1) / share - w0) + 1;
    slot0[parts] = (int64_t)v_pre * a.Hkv + kvh + w0;
    col0[parts] = (mi - sub * a.M) * G;
    ++parts;
  }
  // output row of column r: query token r / G, head kvh * G + r % G of sequence b
  auto out_row = [&](int r) { return (((int64_t)b * a.Qn + r / G) * a.Hq + (int64_t)kvh * G + r % G) * D; };
  if (parts == 0) {
    const int nz = (ncol - cbase < 16 ? ncol - cbase : 16) * D;
    for (int i = tid; i < nz; i += kCombineThreads) {
      const int64_t at = out_row(cbase + i / D) + i % D;
      if constexpr (OUT_BF16) static_cast<uint16_t*>(a.out)[at] = 0;
      else static_cast<float*>(a.out)[at] = 0.f;
    }
    return;
  }
  if (parts == 1 && nseg[0] == 1 && own_may_final) return;  // one chunk wrote the output

  // thread t owns column h = cbase + t / 16 (if < ncol) and dims [ (t % 16) * D/16, +D/16 )
  constexpr int DE = D / 16;
  const int h = cbase + (tid >> 4);
  const int d0 = (tid & 15) * DE;
  if (h >= ncol) return;
  float acc[DE];
#pragma unroll
  for (int e = 0; e < DE; ++e) acc[e] = 0.f;
  float M = kNegInf, den = 0.f;
  // the parts' segments as one list (part 0 first), so a sequence with few
  // segments in all takes one round trip whatever entries they come from
  const int n0 = nseg[0];
  const int ntot = n0 + (parts > 1 ? nseg[1] : 0);
  {
    for (int s0 = 0; s0 < ntot; s0 += kCombineChunk) {
      const int ns = ntot - s0 < kCombineChunk ? ntot - s0 : kCombineChunk;
      float vm[kCombineChunk], vl[kCombineChunk];
      f32x4 va[kCombineChunk][DE / 4];
#pragma unroll
      for (int q = 0; q < kCombineChunk; ++q) {
        const bool live = q < ns;
        const int k = s0 + (live ? q : 0);
        const int part = k < n0 ? 0 : 1;
        const int64_t at = (slot0[part] + (k - (part ? n0 : 0))) * a.Gp + col0[part] + h;
        vm[q] = live ? a.ws_m[at] : kNegInf;
        vl[q] = live ? a.ws_l[at] : 0.f;
        const f32x4* row = reinterpret_cast<const f32x4*>(a.ws_acc + at * D + d0);
#pragma unroll
        for (int e = 0; e < DE / 4; ++e) va[q][e] = live ? row[e] : f32x4{0.f, 0.f, 0.f, 0.f};
      }
      float mc = M;
#pragma unroll
      for (int q = 0; q < kCombineChunk; ++q) mc = fmaxf(mc, vm[q]);
      const float ms = mc == kNegInf ? 0.f : mc;
      const float r = fast_exp2((M == kNegInf ? ms : M) - ms);
      den *= r;
#pragma unroll
      for (int e = 0; e < DE; ++e) acc[e] *= r;
#pragma unroll
      for (int q = 0; q < kCombineChunk; ++q) {
        const float w = fast_exp2(vm[q] - ms);  // 0 for padded segments (m = -inf)
        den = fmaf(w, vl[q], den);
#pragma unroll
        for (int e = 0; e < DE / 4; ++e) {
          acc[4 * e] = fmaf(w, va[q][e][0], acc[4 * e]);
          acc[4 * e + 1] = fmaf(w, va[q][e][1], acc[4 * e + 1]);
          acc[4 * e + 2] = fmaf(w, va[q][e][2], acc[4 * e + 2]);
          acc[4 * e + 3] = fmaf(w, va[q][e][3], acc[4 * e + 3]);
        }
      }
      M = mc;
    }
  }
  const float inv = den > 0.f ? 1.f / den : 0.f;
  const int64_t o = out_row(h) + d0;
#pragma unroll
  for (int e = 0; e < DE; ++e) {
    if constexpr (OUT_BF16) static_cast<uint16_t*>(a.out)[o + e] = (uint16_t)f32_to_bf16_bits(acc[e] * inv);
    else static_cast<float*>(a.out)[o + e] = acc[e] * inv;
  }
}

// ------------------------------------------------------------- shared prefix

// Shared-prefix mode, before the decode kernel: the number of leading blocks
// group g's members really share. It is at most the caller's bound, at most
// every member's full blocks, and only as long as every member's block-table
// row holds the same ids, so a wrong bound costs speed, never correctness (a
// bound cut short by differing ids is flagged). One workgroup per group: each
// thread compares one block position across the members, 8 loads in flight.
constexpr int kPrefixThreads = 256;

__device__ __forceinline__ int block_min(int x, int* red) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    const int y = __shfl_xor(x, o, 64);
    x = x < y ? x : y;
  }
  __syncthreads();  // red is reused: earlier readers are done
  if (lane_id() == 0) red[threadIdx.x >> 6] = x;
  __syncthreads();
#pragma unroll
  for (int w = 0; w < kPrefixThreads / 64; ++w) x = x < red[w] ? x : red[w];
  return x;
}

__global__ __launch_bounds__(kPrefixThreads) void prefix_kernel(DecodeArgs a) {  // grid: one workgroup per group
  __shared__ int red[kPrefixThreads / 64];
  const int g = blockIdx.x;
  const int tid = threadIdx.x;
  const int gs = a.group_size, first = g * gs;
  int S = a.shared_blocks[g];
  S = S < 0 ? 0 : (S > a.max_blocks ? a.max_blocks : S);
  for (int i = tid; i < gs; i += kPrefixThreads) {
    const int full = clamp_len(a, a.seq_lens[first + i]) / kBlockSize;
    S = S < full ? S : full;
  }
  S = block_min(S, red);
  const int32_t* row0 = a.block_table + (int64_t)first * a.max_blocks;
  int common = S;
  for (int j0 = 0; j0 < S; j0 += kPrefixThreads) {
    const int j = j0 + tid;
    bool same = true;
    if (j < S) {
      const int id = row0[j];
      for (int i = 1; i < gs; i += 8) {
        int v[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
          v[u] = i + u < gs ? a.block_table[(int64_t)(first + i + u) * a.max_blocks + j] : id;
#pragma unroll
        for (int u = 0; u < 8; ++u) same &= v[u] == id;
      }
    }
    const int d = block_min(j < S && !same ? j : INT32_MAX, red);
    if (d != INT32_MAX) {
      common = d;
      break;
    }
  }
  if (tid == 0) {
    a.sg[g] = common;
    if (common < S) atomicOr(a.hdr + kHdrStatus, kStatusPrefixShortened);
  }
}

// ------------------------------------------------------------- dispatch

template <Variant V, KvType KV, int D, int GV>
void* kernel_ptr() {
  // the two-tile body of the wide kernel does not fit two fp8 waves per SIMD
  if constexpr (V == Variant::Mfma && KV == KvType::FP8 && GV != kWideColumns)
    return reinterpret_cast<void*>(&decode_kernel_occ2<V, KV, D, GV>);
  else if constexpr (V == Variant::Mfma) return reinterpret_cast<void*>(&decode_kernel<V, KV, D, GV>);
  else return reinterpret_cast<void*>(&decode_kernel_vec<V, KV, D, GV>);
}

template <Variant V, KvType KV, int D>
void* pick_g(int G, bool wide) {
  if constexpr (V == Variant::Mfma) {
    return wide ? kernel_ptr<V, KV, D, kWideColumns>() : kernel_ptr<V, KV, D, 16>();
  } else {
    if (G <= 1) return kernel_ptr<V, KV, D, 1>();
    if (G <= 2) return kernel_ptr<V, KV, D, 2>();
    if (G <= 4) return kernel_ptr<V, KV, D, 4>();
    return kernel_ptr<V, KV, D, 8>();
  }
}

template <Variant V, KvType KV>
void* pick_d(int D, int G, bool wide) {
  return D == 64 ? pick_g<V, KV, 64>(G, wide) : pick_g<V, KV, 128>(G, wide);
}

void* pick(Variant v, KvType kv, int D, int G, bool wide) {
  if (v == Variant::Mfma) {
    if (kv == KvType::BF16) return pick_d<Variant::Mfma, KvType::BF16>(D, G, wide);
    if (kv == KvType::FP8) return pick_d<Variant::Mfma, KvType::FP8>(D, G, wide);
    return nullptr;
  }
  if (wide) return nullptr;
  if (kv == KvType::F32) return pick_d<Variant::Vector, KvType::F32>(D, G, false);
  if (kv == KvType::BF16) return pick_d<Variant::Vector, KvType::BF16>(D, G, false);
  return pick_d<Variant::Vector, KvType::FP8>(D, G, false);
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, Variant v, KvType kv, hipStream_t s) {
  void* fn = pick(v, kv, a.D, a.G, a.Gp > 16);
  if (!fn) return hipErrorInvalidValue;
  DecodeArgs args = a;
  const void* q = a.q;
  const void* kc = a.k_cache;
  const void* vc = a.v_cache;
  const int32_t* bt = a.block_table;
  const int32_t* lens = a.seq_lens;
  const float* scales = a.kv_scales;
  void* params[] = {&args, &q, &kc, &vc, &bt, &lens, &scales};
  const int wpg = a.waves_per_group;
  return hipLaunchKernel(fn, dim3(a.waves / wpg), dim3(64 * wpg), params, 0, s);
}

hipError_t launch_combine(const DecodeArgs& a, hipStream_t s) {
  void* fn;
  if (a.out_bf16)
    fn = a.D == 64 ? reinterpret_cast<void*>(&combine_kernel<true, 64>)
                   : reinterpret_cast<void*>(&combine_kernel<true, 128>);
  else
    fn = a.D == 64 ? reinterpret_cast<void*>(&combine_kernel<false, 64>)
                   : reinterpret_cast<void*>(&combine_kernel<false, 128>);
  const unsigned units = (unsigned)a.B * (unsigned)a.Hkv;
  if (units == 0) return hipSuccess;
  const unsigned halves = (unsigned)(a.Qn * a.G + 15) / 16;  // 16 columns per workgroup
  DecodeArgs args = a;
  void* params[] = {&args};
  return hipLaunchKernel(fn, dim3(units, halves), dim3(kCombineThreads), params, 0, s);
}

hipError_t launch_prefix(const DecodeArgs& a, int num_groups, hipStream_t s) {
  if (num_groups <= 0) return hipSuccess;
  DecodeArgs args = a;
  void* params[] = {&args};
  return hipLaunchKernel(reinterpret_cast<void*>(&prefix_kernel), dim3(num_groups), dim3(kPrefixThreads), params, 0,
                         s);
}

hipError_t decode_occupancy(Variant v, KvType kv, int D, int G, bool wide, int* waves_per_cu) {
  void* fn = pick(v, kv, D, G, wide);
  if (!fn) return hipErrorInvalidValue;
  int wgs = 0;
  const hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&wgs, fn, 64, 0);
  *waves_per_cu = wgs;
  return e;
}

}  // namespace pda
