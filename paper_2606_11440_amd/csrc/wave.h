// Wavefront primitives for gfx950 (64-lane waves).
//
// Ballot / prefix counts (mbcnt), cross-lane exchanges, a 64-lane bitonic
// sort network on 64-bit keys, and fp32 -> bf16 round-to-nearest-even.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace im {

constexpr int kWave = 64;

__device__ __forceinline__ int lane_id() { return __lane_id(); }

// 64-bit mask of lanes where pred holds.
__device__ __forceinline__ uint64_t ballot(bool pred) { return __ballot(pred); }

// Number of set bits of `mask` strictly below this lane.
__device__ __forceinline__ int prefix_count(uint64_t mask) {
  uint32_t lo = (uint32_t)mask, hi = (uint32_t)(mask >> 32);
  return (int)__builtin_amdgcn_mbcnt_hi(hi, __builtin_amdgcn_mbcnt_lo(lo, 0u));
}

__device__ __forceinline__ int popc64(uint64_t m) { return __popcll(m); }

// Position of the r-th (0-based) set bit of m; m must have more than r bits.
__device__ __forceinline__ int nth_set_bit(uint64_t m, int r) {
  int pos = 0;
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    uint64_t low = m & ((w == 64) ? ~0ull : ((1ull << w) - 1ull));
    int c = __popcll(low);
    if (r >= c) { r -= c; m >>= w; pos += w; }
    else { m = low; }
  }
  return pos;
}

__device__ __forceinline__ int32_t shfl(int32_t v, int src) { return __shfl(v, src, kWave); }
__device__ __forceinline__ int64_t shfl(int64_t v, int src) {
  int32_t lo = __shfl((int32_t)(uint32_t)v, src, kWave);
  int32_t hi = __shfl((int32_t)(v >> 32), src, kWave);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}
// Value of a 64-bit variable in lane `src` (wave-uniform result).
__device__ __forceinline__ int64_t readlane64(int64_t v, int src) {
  const uint32_t lo = __builtin_amdgcn_readlane((int32_t)(uint32_t)v, src);
  const uint32_t hi = __builtin_amdgcn_readlane((int32_t)(v >> 32), src);
  return (int64_t)(((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ int32_t shfl_xor(int32_t v, int m) { return __shfl_xor(v, m, kWave); }
__device__ __forceinline__ int64_t shfl_xor(int64_t v, int m) {
  int32_t lo = __shfl_xor((int32_t)(uint32_t)v, m, kWave);
  int32_t hi = __shfl_xor((int32_t)(v >> 32), m, kWave);
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Wave-wide sums (every lane gets the result).
__device__ __forceinline__ int64_t wave_sum(int64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}
__device__ __forceinline__ uint64_t wave_or(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v |= (uint64_t)shfl_xor((int64_t)v, m);
  return v;
}

// Value of v in lane (lane ^ S), S a power of two up to 32, with no LDS
// traffic: DPP moves inside rows of 16 lanes, the gfx950 permlane swaps
// across rows. Every lane of the wave must be active.
template <int S>
__device__ __forceinline__ int32_t xshfl(int32_t v) {
  static_assert(S == 1 || S == 2 || S == 4 || S == 8 || S == 16 || S == 32, "xor distance");
  if constexpr (S == 1) {
    return __builtin_amdgcn_update_dpp(0, v, 0xB1, 0xf, 0xf, false);    // quad_perm [1,0,3,2]
  } else if constexpr (S == 2) {
    return __builtin_amdgcn_update_dpp(0, v, 0x4E, 0xf, 0xf, false);    // quad_perm [2,3,0,1]
  } else if constexpr (S == 4) {
    // i ^ 4 == 7 - (i ^ 3) inside each 8 lanes: quad_perm [3,2,1,0], then half-row mirror
    const int32_t r = __builtin_amdgcn_update_dpp(0, v, 0x1B, 0xf, 0xf, false);
    return __builtin_amdgcn_update_dpp(0, r, 0x141, 0xf, 0xf, false);
  } else if constexpr (S == 8) {
    return __builtin_amdgcn_update_dpp(0, v, 0x128, 0xf, 0xf, false);   // row_ror:8
  } else if constexpr (S == 16) {
    // swap(odd rows of a, even rows of b) with a = b = v: a' = rows (0,0,2,2), b' = (1,1,3,3)
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return (lane_id() & 16) ? (int32_t)r[0] : (int32_t)r[1];
  } else {
    // swap(upper half of a, lower half of b): a' = (lo, lo), b' = (hi, hi)
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (lane_id() & 32) ? (int32_t)r[0] : (int32_t)r[1];
  }
}
template <int S>
__device__ __forceinline__ int64_t xshfl(int64_t v) {
  const int32_t lo = xshfl<S>((int32_t)(uint32_t)v);
  const int32_t hi = xshfl<S>((int32_t)(v >> 32));
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// One compare-exchange stage of a bitonic network at xor distance S: this
// lane keeps the smaller key if it is the low end of an ascending pair.
template <int S, int NP>
__device__ __forceinline__ void cmpx(int64_t& k, int32_t (&p)[NP], bool ascending) {
  const int64_t pk = xshfl<S>(k);
  int32_t pp[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) pp[i] = xshfl<S>(p[i]);
  // The lane takes its partner's key when that is the smaller one (low end
  // of an ascending pair) or the larger one (otherwise). For distinct keys
  // "larger" is "not smaller"; equal keys only occur as padding, whose
  // payloads are never used, so one compare and a flip suffice.
  const bool flip = ((lane_id() & S) != 0) == ascending;
  const bool take = (pk < k) != flip;
  // selects, not a branch: the whole network stays straight-line code
  k = take ? pk : k;
#pragma unroll
  for (int i = 0; i < NP; ++i) p[i] = take ? pp[i] : p[i];
}

// Ascending sort of a bitonic sequence of 64 keys (a half-cleaner cascade).
template <int NP>
__device__ __forceinline__ void bitonic_merge64(int64_t& k, int32_t (&p)[NP]) {
  cmpx<32, NP>(k, p, true);
  cmpx<16, NP>(k, p, true);
  cmpx<8, NP>(k, p, true);
  cmpx<4, NP>(k, p, true);
  cmpx<2, NP>(k, p, true);
  cmpx<1, NP>(k, p, true);
}

// Merge stages of block size SIZE: ascending where lane & SIZE is 0 (or for
// the full 64), descending otherwise.
template <int SIZE, int NP>
__device__ __forceinline__ void bitonic_block(int64_t& k, int32_t (&p)[NP]) {
  const bool asc = SIZE == kWave || (lane_id() & SIZE) == 0;
  if constexpr (SIZE >= 64) cmpx<32, NP>(k, p, asc);
  if constexpr (SIZE >= 32) cmpx<16, NP>(k, p, asc);
  if constexpr (SIZE >= 16) cmpx<8, NP>(k, p, asc);
  if constexpr (SIZE >= 8) cmpx<4, NP>(k, p, asc);
  if constexpr (SIZE >= 4) cmpx<2, NP>(k, p, asc);
  cmpx<1, NP>(k, p, asc);
}

// Ascending bitonic sort of 64 keys (one per lane), payload carried along.
template <int NP>
__device__ __forceinline__ void bitonic_sort64(int64_t& k, int32_t (&p)[NP]) {
  bitonic_block<2, NP>(k, p);
  bitonic_block<4, NP>(k, p);
  bitonic_block<8, NP>(k, p);
  bitonic_block<16, NP>(k, p);
  bitonic_block<32, NP>(k, p);
  bitonic_block<64, NP>(k, p);
}

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __uint_as_float((uint32_t)h << 16);
}

}  // namespace im
