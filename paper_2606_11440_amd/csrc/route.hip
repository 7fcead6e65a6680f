// Route step of the tick: feature gather, policy MLP on MFMA, masked argmax.
//
// Sec. 3 Eq. 1 (the executor's state), Sec. 3 "Action" (a -> model a / K,
// depth a % K) and Sec. 4.2 (a policy network scores every joint action; it
// is deployed greedily here). One wave owns 32 request rows; a block holds 4
// waves (128 rows).
//
// The MLP is evaluated transposed, Y^T = W X^T, on 32x32 MFMA tiles: the
// weights are the A operand (streamed from L2, pre-packed so that each lane
// reads 16 contiguous bytes per instruction) and the activations are the B
// operand. The accumulator layout of one layer (lane = row n + 32 g, register v
// holds output feature 8(v/4) + 4g + v%4 of its tile) is used directly as the
// B operand of the next layer; the next layer's weight columns are permuted at
// pool creation to match, so activations never leave registers.
//
// bf16 pools use v_mfma_f32_32x32x16_bf16 (fp32 accumulate, hidden activations
// rounded to bf16 after the ReLU); fp32 pools use v_mfma_f32_32x32x2_f32.
#include <math.h>

#include "im_internal.h"
#include "wave.h"

namespace im {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x16 mfma_bf16(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}
__device__ __forceinline__ f32x16 mfma_f32(float a, float b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
}

struct RowCtx {
  int32_t r;        // request row (tail lanes: >= n_total)
  bool live;        // r < n_total
  bool bad_q;       // q_idx out of range
  int32_t e;        // env of the row
  int32_t q;        // embedding row (0 when bad)
  int32_t budget;
  uint64_t amask;   // bit a set when action a is valid
};

__device__ __forceinline__ RowCtx row_setup(const RouteArgs& a, int32_t r) {
  RowCtx c;
  c.r = r;
  c.live = r < a.n_total;
  const int32_t rr = c.live ? r : a.n_total - 1;
  // env: the largest e in [0, E] with offsets[e] <= rr
  int lo = 0, hi = a.E;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.offsets[mid] <= rr) lo = mid; else hi = mid - 1;
  }
  c.e = lo < a.E ? lo : a.E - 1;
  const int32_t q = a.q_idx[rr];
  c.bad_q = q < 0 || (int64_t)q >= a.Q;
  c.q = c.bad_q ? 0 : q;
  c.budget = a.budget[rr];
  // Valid actions: model enabled, c_m > 0 and its queue below capacity.
  const ModelRec* ms = a.ms + (size_t)c.e * a.M;
  const uint64_t kmask = (a.K >= 64) ? ~0ull : ((1ull << a.K) - 1ull);
  uint64_t am = 0;
  for (int m = 0; m < a.M; ++m) {
    const bool ok = ms[m].enabled != 0 && ms[m].cap > 0 && ms[m].qlen < a.qcap;
    if (ok) am |= kmask << (m * a.K);
  }
  c.amask = am;
  return c;
}

// Feature k >= embed_dim of a row: load statistics of the row's env (stat-major:
// queue depth of all models, then busy/c_m, latency EWMA, backlog), then the
// normalised budget, then zeros. Each is one fp32 product of an integer and a
// reciprocal rounded once to fp32 on the host.
__device__ __forceinline__ float tail_feature(const RouteArgs& a, const RowCtx& c, int k,
                                              const float* inv_tab) {
  const int k2 = k - a.embed_dim;
  if (k2 < 4 * a.M) {
    const int s = k2 / a.M;
    const int m = k2 - s * a.M;
    const ModelRec& x = a.ms[(size_t)c.e * a.M + m];
    int cap = x.cap < 0 ? 0 : (x.cap > IM_MAX_SLOTS ? IM_MAX_SLOTS : x.cap);
    switch (s) {
      case 0: return (float)x.qlen * a.inv_qcap;
      case 1: return (float)x.busy * inv_tab[cap];
      case 2: return (float)x.ewma * a.inv_lat;
      default: return (float)x.backlog * inv_tab[IM_MAX_SLOTS + 1 + cap];
    }
  }
  if (k2 == 4 * a.M) return (float)c.budget * a.inv_bud;
  return 0.f;
}

__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  return (uint32_t)f32_to_bf16_rne(lo) | ((uint32_t)f32_to_bf16_rne(hi) << 16);
}

// Layer-1 B fragment of K block kb (bf16): features 16 kb + 8 g + j, j = 0..7.
__device__ __forceinline__ u32x4 gather_bf16(const RouteArgs& a, const RowCtx& c, int kb, int g,
                                             const float* inv_tab) {
  const int k0 = 16 * kb + 8 * g;
  const uint16_t* emb = (const uint16_t*)a.emb;
  if (k0 + 8 <= a.embed_dim && (a.embed_dim & 7) == 0) {
    return *(const u32x4*)(emb + (size_t)c.q * a.embed_dim + k0);
  }
  float f[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const int k = k0 + j;
    f[j] = k < a.embed_dim ? bf16_to_f32(emb[(size_t)c.q * a.embed_dim + k])
                           : tail_feature(a, c, k, inv_tab);
  }
  u32x4 v;
  v.x = pack2(f[0], f[1]);
  v.y = pack2(f[2], f[3]);
  v.z = pack2(f[4], f[5]);
  v.w = pack2(f[6], f[7]);
  return v;
}

// Masked argmax over the lane pair (n, n + 32), logits store, action store.
template <int AT>
__device__ __forceinline__ void epilogue(const RouteArgs& a, const RowCtx& c, f32x16 (&acc)[AT],
                                         const float* bias, int g) {
  float best = 0.f;
  int ba = -1;
#pragma unroll
  for (int T = 0; T < AT; ++T) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int act = 32 * T + 8 * (v >> 2) + 4 * g + (v & 3);
      const float z = acc[T][v] + bias[(T * 2 + g) * 16 + v];
      acc[T][v] = z;
      if (act < a.A && ((c.amask >> act) & 1ull)) {
        if (ba < 0 || z > best) { best = z; ba = act; }
      }
    }
  }
  const float ob = __shfl_xor(best, 32, 64);
  const int oa = __shfl_xor(ba, 32, 64);
  if (oa >= 0 && (ba < 0 || ob > best || (ob == best && oa < ba))) { best = ob; ba = oa; }
  if (!c.live) return;
  if (g == 0) {
    a.actions[c.r] = c.bad_q ? -1 : ba;
    if (c.bad_q) atomicOr(a.err, IM_ERR_QIDX);
  }
  if (a.logits) {
    float* out = a.logits + (size_t)c.r * a.A;
#pragma unroll
    for (int T = 0; T < AT; ++T) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int act = 32 * T + 8 * (v >> 2) + 4 * g + (v & 3);
        if (act < a.A) out[act] = c.bad_q ? 0.f : acc[T][v];
      }
    }
  }
}

// bias + ReLU + bf16 rounding of one accumulator tile into two B fragments.
__device__ __forceinline__ void tile_to_frags(const f32x16& acc, const float* bias, int T, int g,
                                              u32x4& f0, u32x4& f1) {
  float h[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) h[v] = fmaxf(acc[v] + bias[(T * 2 + g) * 16 + v], 0.f);
  f0.x = pack2(h[0], h[1]);   f0.y = pack2(h[2], h[3]);
  f0.z = pack2(h[4], h[5]);   f0.w = pack2(h[6], h[7]);
  f1.x = pack2(h[8], h[9]);   f1.y = pack2(h[10], h[11]);
  f1.z = pack2(h[12], h[13]); f1.w = pack2(h[14], h[15]);
}

template <int H, int NL, int AT>
__global__ __launch_bounds__(256) void route_bf16(RouteArgs a) {
  const float* inv_tab = a.inv_tab;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, g = lane >> 5;
  const int32_t row0 = (int32_t)(blockIdx.x * 4 + wave) * 32;
  if (row0 >= a.n_total) return;
  const RowCtx c = row_setup(a, row0 + n);
  constexpr int TH = H / 32;        // hidden tiles
  constexpr int KH = H / 16;        // K blocks over a hidden layer
  const u32x4* W1 = (const u32x4*)a.W[0];
  f32x16 acc[TH];
#pragma unroll
  for (int T = 0; T < TH; ++T) acc[T] = f32x16{};
  for (int kb = 0; kb < a.k1; ++kb) {
    const u32x4 xb = gather_bf16(a, c, kb, g, inv_tab);
#pragma unroll
    for (int T = 0; T < TH; ++T) acc[T] = mfma_bf16(W1[(T * a.k1 + kb) * 64 + lane], xb, acc[T]);
  }
  u32x4 h1[KH];
#pragma unroll
  for (int T = 0; T < TH; ++T) tile_to_frags(acc[T], a.bias[0], T, g, h1[2 * T], h1[2 * T + 1]);

  f32x16 out[AT];
#pragma unroll
  for (int T = 0; T < AT; ++T) out[T] = f32x16{};
  if constexpr (NL == 2) {
    const u32x4* W2 = (const u32x4*)a.W[1];
#pragma unroll
    for (int kb = 0; kb < KH; ++kb) {
#pragma unroll
      for (int T = 0; T < AT; ++T) out[T] = mfma_bf16(W2[(T * KH + kb) * 64 + lane], h1[kb], out[T]);
    }
    epilogue<AT>(a, c, out, a.bias[1], g);
  } else {
    // Layer 2 in chunks of CH output features; each chunk is consumed by the
    // output layer right away, so only one chunk of h2 is ever live.
    constexpr int CH = H < 128 ? H : 128;
    constexpr int TC = CH / 32;
    const u32x4* W2 = (const u32x4*)a.W[1];
    const u32x4* W3 = (const u32x4*)a.W[2];
    for (int cc = 0; cc < H / CH; ++cc) {
      f32x16 acc2[TC];
#pragma unroll
      for (int T = 0; T < TC; ++T) acc2[T] = f32x16{};
#pragma unroll
      for (int kb = 0; kb < KH; ++kb) {
#pragma unroll
        for (int T = 0; T < TC; ++T)
          acc2[T] = mfma_bf16(W2[((cc * TC + T) * KH + kb) * 64 + lane], h1[kb], acc2[T]);
      }
#pragma unroll
      for (int T = 0; T < TC; ++T) {
        u32x4 f0, f1;
        tile_to_frags(acc2[T], a.bias[1], cc * TC + T, g, f0, f1);
        const int kb3 = (cc * TC + T) * 2;
#pragma unroll
        for (int To = 0; To < AT; ++To) {
          out[To] = mfma_bf16(W3[(To * KH + kb3) * 64 + lane], f0, out[To]);
          out[To] = mfma_bf16(W3[(To * KH + kb3 + 1) * 64 + lane], f1, out[To]);
        }
      }
    }
    epilogue<AT>(a, c, out, a.bias[2], g);
  }
}

template <int H, int NL, int AT>
__global__ __launch_bounds__(256) void route_f32(RouteArgs a) {
  const float* inv_tab = a.inv_tab;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, g = lane >> 5;
  const int32_t row0 = (int32_t)(blockIdx.x * 4 + wave) * 32;
  if (row0 >= a.n_total) return;
  const RowCtx c = row_setup(a, row0 + n);
  constexpr int TH = H / 32;
  constexpr int KH = H / 2;         // 2-wide K steps over a hidden layer
  const float* W1 = (const float*)a.W[0];
  const float* emb = (const float*)a.emb;
  f32x16 acc[TH];
#pragma unroll
  for (int T = 0; T < TH; ++T) acc[T] = f32x16{};
  for (int i = 0; i < a.k1; ++i) {
    const int k = 2 * i + g;
    const float x = k < a.embed_dim ? emb[(size_t)c.q * a.embed_dim + k]
                                    : tail_feature(a, c, k, inv_tab);
#pragma unroll
    for (int T = 0; T < TH; ++T) acc[T] = mfma_f32(W1[(T * a.k1 + i) * 64 + lane], x, acc[T]);
  }
#pragma unroll
  for (int T = 0; T < TH; ++T) {
#pragma unroll
    for (int v = 0; v < 16; ++v) acc[T][v] = fmaxf(acc[T][v] + a.bias[0][(T * 2 + g) * 16 + v], 0.f);
  }
  f32x16 out[AT];
#pragma unroll
  for (int T = 0; T < AT; ++T) out[T] = f32x16{};
  if constexpr (NL == 2) {
    const float* W2 = (const float*)a.W[1];
#pragma unroll
    for (int i = 0; i < KH; ++i) {
#pragma unroll
      for (int T = 0; T < AT; ++T)
        out[T] = mfma_f32(W2[(T * KH + i) * 64 + lane], acc[i >> 4][i & 15], out[T]);
    }
    epilogue<AT>(a, c, out, a.bias[1], g);
  } else {
    constexpr int CH = H < 128 ? H : 128;
    constexpr int TC = CH / 32;
    const float* W2 = (const float*)a.W[1];
    const float* W3 = (const float*)a.W[2];
    for (int cc = 0; cc < H / CH; ++cc) {
      f32x16 acc2[TC];
#pragma unroll
      for (int T = 0; T < TC; ++T) acc2[T] = f32x16{};
#pragma unroll
      for (int i = 0; i < KH; ++i) {
#pragma unroll
        for (int T = 0; T < TC; ++T)
          acc2[T] = mfma_f32(W2[((cc * TC + T) * KH + i) * 64 + lane], acc[i >> 4][i & 15], acc2[T]);
      }
#pragma unroll
      for (int T = 0; T < TC; ++T) {
        const int Tg = cc * TC + T;
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const float h = fmaxf(acc2[T][v] + a.bias[1][(Tg * 2 + g) * 16 + v], 0.f);
          const int i3 = 16 * Tg + v;
#pragma unroll
          for (int To = 0; To < AT; ++To)
            out[To] = mfma_f32(W3[(To * KH + i3) * 64 + lane], h, out[To]);
        }
      }
    }
    epilogue<AT>(a, c, out, a.bias[2], g);
  }
}

typedef void (*RouteKernel)(RouteArgs);

template <int H, int NL>
RouteKernel pick_bf16(int at) { return at == 1 ? route_bf16<H, NL, 1> : route_bf16<H, NL, 2>; }
template <int H, int NL>
RouteKernel pick_f32(int at) { return at == 1 ? route_f32<H, NL, 1> : route_f32<H, NL, 2>; }

template <int NL>
RouteKernel pick(int dtype, int hidden, int at) {
  if (dtype == IM_BF16) {
    switch (hidden) {
      case 32: return pick_bf16<32, NL>(at);
      case 64: return pick_bf16<64, NL>(at);
      case 128: return pick_bf16<128, NL>(at);
      case 256: return pick_bf16<256, NL>(at);
      case 512: return pick_bf16<512, NL>(at);
    }
  } else {
    switch (hidden) {
      case 32: return pick_f32<32, NL>(at);
      case 64: return pick_f32<64, NL>(at);
      case 128: return pick_f32<128, NL>(at);
      case 256: return pick_f32<256, NL>(at);
    }
  }
  return nullptr;
}

}  // namespace

bool route_supported(int dtype, int hidden, int n_layers, int out_tiles) {
  if (out_tiles < 1 || out_tiles > 2) return false;
  RouteKernel k = n_layers == 2 ? pick<2>(dtype, hidden, out_tiles)
                 : n_layers == 3 ? pick<3>(dtype, hidden, out_tiles) : nullptr;
  return k != nullptr;
}

hipError_t launch_route(const RouteArgs& a, int dtype, int hidden, int n_layers, int out_tiles,
                        hipStream_t s) {
  RouteKernel k = nullptr;
  if (out_tiles >= 1 && out_tiles <= 2) {
    if (n_layers == 2) k = pick<2>(dtype, hidden, out_tiles);
    else if (n_layers == 3) k = pick<3>(dtype, hidden, out_tiles);
  }
  if (!k) return hipErrorInvalidValue;
  if (a.n_total <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((a.n_total + 127) / 128);
  hipLaunchKernelGGL(k, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace im
