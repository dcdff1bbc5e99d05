// HIP kernel that appends one decode step's new keys and values to the paged
// KV cache on MI355X (gfx950).
//
// Every rollout decode step (the paper's Sec. 2.2) produces one token per
// live sequence; its key and value go into the sequence's paged cache (the
// vLLM block layout the paper cites in Sec. 8) before attention reads it.
// Token t of sequence b lands in block block_table[b, t / 16], slot t % 16:
// a row of the token-major K tile [16][D] and a column of the dim-major V tile
// [D][16].
//
// fp8 (OCP E4M3) caches keep one scale per (block, KV head) tile and per K / V
// at max(amax / 448, 2^-126) over the tokens written to the tile so far, so a
// full tile ends with the per-tile amax scale. A token whose amax exceeds
// 448 * scale raises the scale to its own amax / 448 and re-encodes the tile's
// earlier codes (decoded value * old / new); otherwise only the new token is
// encoded. Slot 0 always starts a fresh scale. Every step that decides a code
// is float32 with one rounding per operation (correctly rounded division), and
// E4M3 encoding rounds to nearest even after clamping to +-448.

#include "pda_internal.h"

#include <stdint.h>

namespace pda {
namespace {

constexpr float kE4M3Max = 448.f;
constexpr float kMinScale = 0x1p-126f;
constexpr int kAppendWaves = 4;  // waves (one per (sequence, KV head)) per workgroup

__device__ __forceinline__ int lane() { return (int)(threadIdx.x & 63); }

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, 64));
  return x;
}

// float32 -> E4M3 code: clamp to +-448, then the hardware conversion (round
// to nearest even).
__device__ __forceinline__ uint8_t enc_e4m3(float z) {
  z = fminf(fmaxf(z, -kE4M3Max), kE4M3Max);
  return (uint8_t)(__builtin_amdgcn_cvt_pk_fp8_f32(z, z, 0, false) & 0xFF);
}

__device__ __forceinline__ float dec_e4m3(uint8_t c) { return __builtin_amdgcn_cvt_f32_fp8((int)c, 0); }

// f32 -> bf16 bits, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t to_bf16(float f) {
  uint32_t u = __builtin_bit_cast(uint32_t, f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Element (token i, dim d) of tile `tile`: K tiles are [16][D], V tiles [D][16].
template <int D>
__device__ __forceinline__ int64_t tile_elem(bool v, int64_t tile, int i, int d) {
  return v ? (tile * D + d) * kBlockSize + i : (tile * kBlockSize + i) * D + d;
}

template <KvType KV, int D>
__global__ __launch_bounds__(64 * kAppendWaves) void append_kernel(AppendArgs a) {
  const int w = blockIdx.x * kAppendWaves + (int)(threadIdx.x >> 6);
  if (w >= a.B * a.Hkv) return;
  const int b = w / a.Hkv, h = w - b * a.Hkv;
  const int t = a.positions[b];
  if (t < 0) return;
  if (t >= kBlockSize * a.max_blocks) {
    if (lane() == 0) atomicOr(a.status, kStatusLenClamped);
    return;
  }
  const int p = a.block_table[(int64_t)b * a.max_blocks + t / kBlockSize];
  if ((unsigned)p >= (uint64_t)a.num_blocks) {
    if (lane() == 0) atomicOr(a.status, kStatusBadBlock);
    return;
  }
  const int o = t % kBlockSize;
  const int64_t tile = (int64_t)p * a.Hkv + h;
  constexpr int E = D / 64;  // elements per lane

  // every input first (K and V values, fp8 scales): the cache stores below may
  // alias them as far as the compiler knows, and would otherwise serialise them
  const int64_t src = ((int64_t)b * a.Hkv + h) * D;
  float x[2][E];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
#pragma unroll
    for (int e = 0; e < E; ++e) {
      const int d = lane() + 64 * e;
      if (a.new_bf16) {
        const uint16_t u = static_cast<const uint16_t*>(c ? a.v_new : a.k_new)[src + d];
        x[c][e] = __builtin_bit_cast(float, (uint32_t)u << 16);
      } else {
        x[c][e] = static_cast<const float*>(c ? a.v_new : a.k_new)[src + d];
      }
    }
  }

  if constexpr (KV != KvType::FP8) {
#pragma unroll
    for (int c = 0; c < 2; ++c) {
#pragma unroll
      for (int e = 0; e < E; ++e) {
        const int64_t at = tile_elem<D>(c == 1, tile, o, lane() + 64 * e);
        if constexpr (KV == KvType::F32) static_cast<float*>(c ? a.v_cache : a.k_cache)[at] = x[c][e];
        else static_cast<uint16_t*>(c ? a.v_cache : a.k_cache)[at] = to_bf16(x[c][e]);
      }
    }
  } else {
    float* sp[2] = {a.kv_scales + tile, a.kv_scales + a.num_blocks * a.Hkv + tile};
    float old[2], amax[2];
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      old[c] = o > 0 ? *sp[c] : 0.f;
      float m = 0.f;
#pragma unroll
      for (int e = 0; e < E; ++e) m = fmaxf(m, fabsf(x[c][e]));
      amax[c] = wave_max(m);
    }
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const bool is_v = c == 1;
      uint8_t* cb = static_cast<uint8_t*>(is_v ? a.v_cache : a.k_cache);
      const bool keep = o > 0 && old[c] > 0.f && amax[c] <= kE4M3Max * old[c];
      float s = old[c];
      if (!keep) {
        s = fmaxf(__fdiv_rn(amax[c], kE4M3Max), kMinScale);
        // re-encode the tile's earlier tokens with the grown scale
        for (int k = lane(); k < o * D; k += 64) {
          const int i = k / D, d = k - i * D;
          const int64_t at = tile_elem<D>(is_v, tile, i, d);
          cb[at] = enc_e4m3(__fdiv_rn(dec_e4m3(cb[at]) * old[c], s));
        }
      }
#pragma unroll
      for (int e = 0; e < E; ++e)
        cb[tile_elem<D>(is_v, tile, o, lane() + 64 * e)] = enc_e4m3(__fdiv_rn(x[c][e], s));
      if (lane() == 0) *sp[c] = s;
    }
  }
}

template <KvType KV>
void* append_for_d(int D) {
  return D == 64 ? reinterpret_cast<void*>(&append_kernel<KV, 64>) : reinterpret_cast<void*>(&append_kernel<KV, 128>);
}

}  // namespace

hipError_t launch_append(const AppendArgs& a, KvType kv, hipStream_t s) {
  const int64_t waves = (int64_t)a.B * a.Hkv;
  if (waves == 0) return hipSuccess;
  void* fn = kv == KvType::F32 ? append_for_d<KvType::F32>(a.D)
             : kv == KvType::BF16 ? append_for_d<KvType::BF16>(a.D)
                                  : append_for_d<KvType::FP8>(a.D);
  AppendArgs args = a;
  void* params[] = {&args};
  return hipLaunchKernel(fn, dim3((unsigned)((waves + kAppendWaves - 1) / kAppendWaves)), dim3(64 * kAppendWaves),
                         params, 0, s);
}

}  // namespace pda
