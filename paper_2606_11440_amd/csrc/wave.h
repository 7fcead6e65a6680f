// Wavefront primitives for gfx950 (64-lane waves).
//
// Ballot / prefix counts (mbcnt), cross-lane exchanges, a 64-lane bitonic
// sort network on 32- or 64-bit keys, and fp32 -> bf16 round-to-nearest-even.
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
// across rows. Every lane of the wave must be active. Every source lane of
// these patterns is a valid lane of the same row, so the DPP "old" operand is
// never used: the moves are issued without one (no initialising move).
template <int CTRL>
__device__ __forceinline__ int32_t dpp(int32_t v) {
  return __builtin_amdgcn_mov_dpp(v, CTRL, 0xf, 0xf, true);
}

template <int S>
__device__ __forceinline__ int32_t xshfl(int32_t v) {
  static_assert(S == 1 || S == 2 || S == 4 || S == 8 || S == 16 || S == 32, "xor distance");
  if constexpr (S == 1) {
    return dpp<0xB1>(v);                 // quad_perm [1,0,3,2]
  } else if constexpr (S == 2) {
    return dpp<0x4E>(v);                 // quad_perm [2,3,0,1]
  } else if constexpr (S == 4) {
    // i ^ 4 == 7 - (i ^ 3) inside each 8 lanes: quad_perm [3,2,1,0], then half-row mirror
    return dpp<0x141>(dpp<0x1B>(v));
  } else if constexpr (S == 8) {
    return dpp<0x128>(v);                // row_ror:8
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
__device__ __forceinline__ uint32_t xshfl(uint32_t v) { return (uint32_t)xshfl<S>((int32_t)v); }
template <int S>
__device__ __forceinline__ int64_t xshfl(int64_t v) {
  const int32_t lo = xshfl<S>((int32_t)(uint32_t)v);
  const int32_t hi = xshfl<S>((int32_t)(v >> 32));
  return (int64_t)(((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// Both halves of a 16-row (S = 16) or 32-lane (S = 32) exchange of v, from
// one permlane swap of v with a copy of itself: lanes in the lower group of
// each pair hold their own value in x and the partner's in y, lanes in the
// upper group the other way round.
//   permlane16_swap(a, b): a' = rows (a0, b0, a2, b2), b' = (a1, b1, a3, b3)
//   permlane32_swap(a, b): a' = (a.lo, b.lo),        b' = (a.hi, b.hi)
template <int S>
__device__ __forceinline__ void swap_halves(int32_t v, int32_t& x, int32_t& y) {
  if constexpr (S == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    x = (int32_t)r[0];
    y = (int32_t)r[1];
  } else {
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    x = (int32_t)r[0];
    y = (int32_t)r[1];
  }
}

// One compare-exchange stage of a bitonic network at xor distance S: this
// lane keeps the smaller key if it is the low end of an ascending pair.
template <int S, int NP, typename KT>
__device__ __forceinline__ void cmpx(KT& k, int32_t (&p)[NP], bool ascending) {
  // The lane takes its partner's key when that is the smaller one (low end
  // of an ascending pair) or the larger one (otherwise). For distinct keys
  // "larger" is "not smaller"; equal keys only occur as padding, whose
  // payloads are never used, so one compare and a flip suffice.
  const bool upper = (lane_id() & S) != 0;
  const bool flip = upper == ascending;
  if constexpr (S >= 16) {
    // x/y hold (own, partner) in lower lanes and (partner, own) in upper
    // lanes; the lane keeps y when (y < x) != flip, i.e. whichever of the two
    // the comparison picks, with no second copy of the key.
    KT kx, ky;
    if constexpr (sizeof(KT) == 8) {
      int32_t xl, yl, xh, yh;
      swap_halves<S>((int32_t)(uint32_t)k, xl, yl);
      swap_halves<S>((int32_t)((uint64_t)k >> 32), xh, yh);
      kx = (KT)(((uint64_t)(uint32_t)xh << 32) | (uint32_t)xl);
      ky = (KT)(((uint64_t)(uint32_t)yh << 32) | (uint32_t)yl);
    } else {
      int32_t x, y;
      swap_halves<S>((int32_t)k, x, y);
      kx = (KT)x;
      ky = (KT)y;
    }
    const bool pick_y = (ky < kx) != flip;
    k = pick_y ? ky : kx;
#pragma unroll
    for (int i = 0; i < NP; ++i) {
      int32_t x, y;
      swap_halves<S>(p[i], x, y);
      p[i] = pick_y ? y : x;
    }
  } else {
    const KT pk = xshfl<S>(k);
    int32_t pp[NP];
#pragma unroll
    for (int i = 0; i < NP; ++i) pp[i] = xshfl<S>(p[i]);
    const bool take = (pk < k) != flip;
    // selects, not a branch: the whole network stays straight-line code
    k = take ? pk : k;
#pragma unroll
    for (int i = 0; i < NP; ++i) p[i] = take ? pp[i] : p[i];
  }
}

// Ascending sort of a bitonic sequence of 64 keys (a half-cleaner cascade).
template <int NP, typename KT>
__device__ __forceinline__ void bitonic_merge64(KT& k, int32_t (&p)[NP]) {
  cmpx<32, NP>(k, p, true);
  cmpx<16, NP>(k, p, true);
  cmpx<8, NP>(k, p, true);
  cmpx<4, NP>(k, p, true);
  cmpx<2, NP>(k, p, true);
  cmpx<1, NP>(k, p, true);
}

// Merge stages of block size SIZE: ascending where lane & SIZE is 0 (or for
// the full 64), descending otherwise.
template <int SIZE, int NP, typename KT>
__device__ __forceinline__ void bitonic_block(KT& k, int32_t (&p)[NP]) {
  const bool asc = SIZE == kWave || (lane_id() & SIZE) == 0;
  if constexpr (SIZE >= 64) cmpx<32, NP>(k, p, asc);
  if constexpr (SIZE >= 32) cmpx<16, NP>(k, p, asc);
  if constexpr (SIZE >= 16) cmpx<8, NP>(k, p, asc);
  if constexpr (SIZE >= 8) cmpx<4, NP>(k, p, asc);
  if constexpr (SIZE >= 4) cmpx<2, NP>(k, p, asc);
  cmpx<1, NP>(k, p, asc);
}

// Ascending bitonic sort of 64 keys (one per lane), payload carried along.
template <int NP, typename KT>
__device__ __forceinline__ void bitonic_sort64(KT& k, int32_t (&p)[NP]) {
  bitonic_block<2, NP>(k, p);
  bitonic_block<4, NP>(k, p);
  bitonic_block<8, NP>(k, p);
  bitonic_block<16, NP>(k, p);
  bitonic_block<32, NP>(k, p);
  bitonic_block<64, NP>(k, p);
}

// Ascending sort of the keys of the first n lanes (n <= 64), over the
// smallest power of two of lanes >= n; keys in the other lanes end up in an
// unspecified order. Fewer stages for short inputs: 6 for n <= 8, 10 for
// n <= 16, 15 for n <= 32, 21 otherwise.
template <typename KT>
__device__ __forceinline__ void bitonic_sort_first(KT& k, int n) {
  int32_t none[1] = {0};   // dead after the network; removed by the compiler
  bitonic_block<2, 1>(k, none);
  if (n <= 2) return;
  bitonic_block<4, 1>(k, none);
  if (n <= 4) return;
  bitonic_block<8, 1>(k, none);
  if (n <= 8) return;
  bitonic_block<16, 1>(k, none);
  if (n <= 16) return;
  bitonic_block<32, 1>(k, none);
  if (n <= 32) return;
  bitonic_block<64, 1>(k, none);
}

// Key-only variants (no payload).
template <typename KT>
__device__ __forceinline__ void bitonic_sort64(KT& k) {
  int32_t none[1] = {0};   // dead after the network; removed by the compiler
  bitonic_sort64<1>(k, none);
}
template <typename KT>
__device__ __forceinline__ void bitonic_merge64(KT& k) {
  int32_t none[1] = {0};
  bitonic_merge64<1>(k, none);
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
