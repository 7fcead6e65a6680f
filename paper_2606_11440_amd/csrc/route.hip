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
// rounded to bf16 after the ReLU); fp32 pools use v_mfma_f32_16x16x4_f32 on
// 16-row tiles in the same transposed scheme.
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
typedef float f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ f32x4 mfma16_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

struct RowCtx {
  int32_t r;        // request row (tail lanes: >= n_total)
  bool live;        // r < n_total
  int32_t bad;      // error bits of the row (IM_ERR_QIDX, IM_ERR_ROLE); 0 when valid
  int32_t e;        // env of the row
  int32_t q;        // embedding row (0 when bad)
  int32_t budget;
  uint64_t amask;   // bit a set when action a is valid
};

// Valid actions of env e: bit a set when model a / K is valid in the env's
// snapshot row (enabled, c_m > 0, queue below capacity).
// The M <= 32 validity bytes start 16-byte aligned (byte 16 M of a row whose
// stride is a multiple of 32 bytes) and the row's padding covers two 16-byte
// words from there, so they arrive in one or two independent loads (a byte
// loop would wait for each byte in turn).
__device__ __forceinline__ uint32_t nonzero_bytes(uint32_t x) {
  // bit i of the result: byte i of x is nonzero (OR-fold each byte into its
  // low bit, then gather bits 0, 8, 16, 24 with one multiply: the shifted
  // copies land on distinct bits, so no carries)
  x |= x >> 4;
  x |= x >> 2;
  x |= x >> 1;
  return ((x & 0x01010101u) * 0x00204081u) >> 21 & 0xfu;
}
__device__ __forceinline__ uint32_t valid_models16(const u32x4 w) {
  return nonzero_bytes(w.x) | nonzero_bytes(w.y) << 4 | nonzero_bytes(w.z) << 8 | nonzero_bytes(w.w) << 12;
}
// The raw validity words of env e (both loaded for every M: the row's padding
// covers them) and the action mask computed from them once they have arrived.
struct ValidRaw {
  u32x4 w0, w1;
};
__device__ __forceinline__ ValidRaw load_valid(const RouteArgs& a, int e) {
  const u32x4* v = (const u32x4*)(a.snap + (size_t)e * snap_stride(a.M) + snap_valid_offset(a.M));
  return {v[0], v[1]};
}
__device__ __forceinline__ uint64_t mask_of(const RouteArgs& a, const ValidRaw& v) {
  uint32_t vm = valid_models16(v.w0);
  if (a.M > 16) vm |= valid_models16(v.w1) << 16;
  if (a.M < 32) vm &= (1u << a.M) - 1u;   // bytes past the M-th are padding
  const uint64_t kmask = (a.K >= 64) ? ~0ull : ((1ull << a.K) - 1ull);
  uint64_t am = 0;
  for (int m = 0; m < a.M; ++m)
    if ((vm >> m) & 1u) am |= kmask << (m * a.K);
  return am;
}
__device__ __forceinline__ uint64_t action_mask(const RouteArgs& a, int e) { return mask_of(a, load_valid(a, e)); }

// Env of rows r[] (per lane) for a wave whose rows lie in [rfirst, rlast]:
// one coalesced load of a 64-entry window of offsets around an interpolated
// guess; a uniform binary search when the guess misses.
__device__ __forceinline__ int32_t find_env_bsearch(const RouteArgs& a, int32_t r) {
  int lo = 0, hi = a.E;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (a.offsets[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo < a.E ? lo : a.E - 1;
}

// First guess of the env window of rows from rfirst on, and its offsets
// (lane i: offsets[e_lo + i]); find_envs_in completes the lookup.
struct EnvWindow {
  int32_t e_lo, ow;
};
__device__ __forceinline__ EnvWindow env_window(const RouteArgs& a, int32_t rfirst) {
  EnvWindow w;
  int32_t e_lo = (int32_t)((float)rfirst * a.envs_per_row) - 16;
  w.e_lo = e_lo < 0 ? 0 : (e_lo > a.E - 1 ? a.E - 1 : e_lo);
  const int32_t wi = w.e_lo + lane_id();
  w.ow = a.offsets[wi < a.E ? wi : a.E];
  return w;
}

template <int NR>
__device__ __forceinline__ void find_envs_in(const RouteArgs& a, EnvWindow w, int32_t rfirst, int32_t rlast,
                                             const int32_t (&r)[NR], int32_t (&e)[NR]) {
  const int lane = lane_id();
  int32_t e_lo = w.e_lo;
  int32_t wi;
  int32_t ow = w.ow;
  bool ok = __builtin_amdgcn_readfirstlane(ow) <= rfirst &&
            rlast < __builtin_amdgcn_readlane(ow, 63);
  if (!ok) {
    e_lo = find_env_bsearch(a, rfirst);
    wi = e_lo + lane;
    ow = a.offsets[wi < a.E ? wi : a.E];
    ok = rlast < __builtin_amdgcn_readlane(ow, 63);
  }
  if (ok) {
    // The window's offsets are ascending. The env of row x is e_lo - 1 plus
    // the number of window offsets <= x: those <= rfirst (one ballot), plus
    // the env boundaries inside the wave's rows (rfirst, rlast], few per wave.
    const int base = e_lo - 1 + popc64(ballot(ow <= rfirst));
#pragma unroll
    for (int j = 0; j < NR; ++j) e[j] = base;
    uint64_t bnd = ballot(ow > rfirst && ow <= rlast);
    while (bnd) {
      const int b = __builtin_ctzll(bnd);
      bnd &= bnd - 1;
      const int32_t ob = __builtin_amdgcn_readlane(ow, b);
#pragma unroll
      for (int j = 0; j < NR; ++j) e[j] += ob <= r[j] ? 1 : 0;
    }
  } else {
#pragma unroll
    for (int j = 0; j < NR; ++j) e[j] = find_env_bsearch(a, r[j] < a.n_total ? r[j] : a.n_total - 1);
  }
#pragma unroll
  for (int j = 0; j < NR; ++j) e[j] = e[j] < 0 ? 0 : (e[j] > a.E - 1 ? a.E - 1 : e[j]);
}

template <int NR>
__device__ __forceinline__ void find_envs(const RouteArgs& a, int32_t rfirst, int32_t rlast,
                                          const int32_t (&r)[NR], int32_t (&e)[NR]) {
  find_envs_in<NR>(a, env_window(a, rfirst), rfirst, rlast, r, e);
}

// Row context of row r (per lane) in a wave whose rows lie in [row0, row0 + 31].
__device__ __forceinline__ RowCtx row_setup(const RouteArgs& a, int32_t row0, int32_t r) {
  RowCtx c;
  c.r = r;
  c.live = r < a.n_total;
  const int32_t rr = c.live ? r : a.n_total - 1;
  const int32_t rl = row0 + 31 < a.n_total ? row0 + 31 : a.n_total - 1;
  const int32_t rows[1] = {rr};
  int32_t env[1];
  find_envs<1>(a, row0, rl, rows, env);
  c.e = env[0];
  const int32_t q = a.q_idx[rr];
  c.bad = (q < 0 || (int64_t)q >= a.Q) ? IM_ERR_QIDX : 0;
  c.q = c.bad ? 0 : q;
  c.budget = a.budget[rr];
  c.amask = action_mask(a, c.e);
  return c;
}

// Row context of row r in env e from its already loaded record fields.
__device__ __forceinline__ RowCtx row_ctx_from(const RouteArgs& a, int32_t r, int32_t e, int32_t q,
                                               int32_t budget) {
  RowCtx c;
  c.r = r;
  c.live = r < a.n_total;
  c.e = e;
  c.bad = (q < 0 || (int64_t)q >= a.Q) ? IM_ERR_QIDX : 0;
  c.q = c.bad ? 0 : q;
  c.budget = budget;
  c.amask = 0;   // set by the caller from load_valid / mask_of
  return c;
}

__device__ __forceinline__ RowCtx row_setup_env(const RouteArgs& a, int32_t r, int32_t e) {
  RowCtx c;
  c.r = r;
  c.live = r < a.n_total;
  const int32_t rr = c.live ? r : a.n_total - 1;
  c.e = e;
  const int32_t q = a.q_idx[rr];
  c.bad = (q < 0 || (int64_t)q >= a.Q) ? IM_ERR_QIDX : 0;
  c.q = c.bad ? 0 : q;
  c.budget = a.budget[rr];
  c.amask = action_mask(a, e);
  return c;
}

// The same, leaving the action mask to the caller (load_valid's words are in
// flight with the row's q_idx and budget).
__device__ __forceinline__ RowCtx row_setup_env_raw(const RouteArgs& a, int32_t r, int32_t e, ValidRaw& vr) {
  RowCtx c;
  c.r = r;
  c.live = r < a.n_total;
  const int32_t rr = c.live ? r : a.n_total - 1;
  c.e = e;
  const int32_t q = a.q_idx[rr];
  c.bad = (q < 0 || (int64_t)q >= a.Q) ? IM_ERR_QIDX : 0;
  c.q = c.bad ? 0 : q;
  c.budget = a.budget[rr];
  vr = load_valid(a, e);
  c.amask = 0;   // mask_of(a, vr) once the words have arrived
  return c;
}

// Feature k >= embed_dim of a row: the env's load statistics (stat-major:
// queue depth of all models, busy/c_m, latency EWMA, backlog; read from the
// snapshot row), then the normalised budget, then zeros.
__device__ __forceinline__ float tail_feature(const RouteArgs& a, const RowCtx& c, int k) {
  const int k2 = k - a.embed_dim;
  if (k2 < 4 * a.M) return a.snap[(size_t)c.e * snap_stride(a.M) + k2];
  if (k2 == 4 * a.M) return (float)c.budget * a.inv_bud;
  return 0.f;
}

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Two fp32 values to packed bf16 (round to nearest even), one
// v_cvt_pk_bf16_f32; element 0 in the low half.
__device__ __forceinline__ uint32_t pack2(float lo, float hi) {
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// ReLU of a float as one integer max on its bits: every negative value
// (and -0) has the sign bit set, so it is below 0 as an int32.
__device__ __forceinline__ float relu(float x) {
  return __int_as_float(max(__float_as_int(x), 0));
}

// bf16(ReLU(lo)), bf16(ReLU(hi)) packed. Rounding to nearest even keeps the
// sign (a negative value rounds to a negative value or -0), so the ReLU is
// applied after rounding, to both halves at once, as a packed signed 16-bit
// max with 0.
__device__ __forceinline__ uint32_t relu_pack2(float lo, float hi) {
  typedef short s16x2 __attribute__((ext_vector_type(2)));
  const s16x2 r = __builtin_bit_cast(s16x2, pack2(lo, hi));
  return __builtin_bit_cast(uint32_t, __builtin_elementwise_max(r, (s16x2){0, 0}));
}

// Layer-1 B fragment of K block kb (bf16): features 16 kb + 8 g + j, j = 0..7.
__device__ __forceinline__ u32x4 gather_bf16(const RouteArgs& a, const RowCtx& c, int kb, int g) {
  const int k0 = 16 * kb + 8 * g;
  const uint16_t* emb = (const uint16_t*)a.emb;
  const bool aligned = (a.embed_dim & 7) == 0;
  if (aligned && k0 + 8 <= a.embed_dim)
    return *(const u32x4*)(emb + (size_t)c.q * a.embed_dim + k0);
  float f[8];
  if (aligned && k0 >= a.embed_dim) {
    // 8 tail features: two aligned float4 loads of the snapshot row, then
    // the budget feature and zero padding selected by index.
    // The row is read only when the block holds a load statistic (k2 < 4M):
    // the 8 floats from k2 then lie inside the row's stride (>= 4M + 9).
    const int k2 = k0 - a.embed_dim;
    float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
    if (k2 < 4 * a.M) {
      const float* row = a.snap + (size_t)c.e * snap_stride(a.M) + k2;
      lo = *(const float4*)row;
      hi = *(const float4*)(row + 4);
    }
    const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    const float fb = (float)c.budget * a.inv_bud;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kk = k2 + j;
      f[j] = kk < 4 * a.M ? v[j] : (kk == 4 * a.M ? fb : 0.f);
    }
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int k = k0 + j;
      f[j] = k < a.embed_dim ? bf16_to_f32(emb[(size_t)c.q * a.embed_dim + k])
                             : tail_feature(a, c, k);
    }
  }
  u32x4 v;
  v.x = pack2(f[0], f[1]);
  v.y = pack2(f[2], f[3]);
  v.z = pack2(f[4], f[5]);
  v.w = pack2(f[6], f[7]);
  return v;
}

// Layer-1 B fragment of K block KB with the embedding width ED known at
// compile time (ED % 16 == 0): each block is either all embedding (one 16-byte
// load) or all tail features (two float4 loads of the snapshot row, then the
// budget feature and zero padding selected by index).
template <int ED, int KB>
__device__ __forceinline__ u32x4 gather_ct(const RouteArgs& a, const RowCtx& c, int g) {
  static_assert(ED % 16 == 0, "embedding width must be a multiple of 16");
  const int k0 = 16 * KB + 8 * g;
  if constexpr (16 * KB + 16 <= ED) {
    const uint16_t* emb = (const uint16_t*)a.emb;
    return *(const u32x4*)(emb + (size_t)c.q * ED + k0);
  } else {
    // the row is read only when the block holds a load statistic (k2 < 4M):
    // the 8 floats from k2 then lie inside the row's stride (>= 4M + 9)
    const int k2 = k0 - ED;
    const int n4 = 4 * a.M;
    float4 lo = make_float4(0.f, 0.f, 0.f, 0.f), hi = lo;
    if (k2 < n4) {
      const float* row = a.snap + (size_t)c.e * snap_stride(a.M) + k2;
      lo = *(const float4*)row;
      hi = *(const float4*)(row + 4);
    }
    const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    const float fb = (float)c.budget * a.inv_bud;
    float f[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int kk = k2 + j;
      f[j] = kk < n4 ? v[j] : (kk == n4 ? fb : 0.f);
    }
    u32x4 r;
    r.x = pack2(f[0], f[1]);
    r.y = pack2(f[2], f[3]);
    r.z = pack2(f[4], f[5]);
    r.w = pack2(f[6], f[7]);
    return r;
  }
}

template <int ED, int KB, int N>
__device__ __forceinline__ void gather_row(const RouteArgs& a, const RowCtx& c, int g, u32x4 (&x)[N]) {
  if constexpr (KB < N) {
    x[KB] = gather_ct<ED, KB>(a, c, g);
    gather_row<ED, KB + 1, N>(a, c, g, x);
  }
}

// Layer-1 B fragments of a row in two steps, so that a wave tile's gather is
// one round trip: gather_issue loads every embedding word and the raw
// snapshot words of the tail blocks (the load statistics; a lane whose block
// starts past them reads from the row's last statistic on, which stays inside
// the row, and ignores the words), gather_finish converts the tail blocks once
// they have arrived (the arithmetic of gather_ct).
template <int ED, int KB1>
struct TailRaw {
  static constexpr int KE = ED / 16 < KB1 ? ED / 16 : KB1;   // K blocks inside the embedding
  static constexpr int KT = KB1 - KE;                          // tail blocks
  float4 t[KT > 0 ? KT : 1][2];
};
template <int ED, int KB1>
__device__ __forceinline__ void gather_issue(const RouteArgs& a, const RowCtx& c, int g, u32x4 (&x)[KB1],
                                             TailRaw<ED, KB1>& raw) {
  static_assert(ED % 16 == 0, "embedding width must be a multiple of 16");
  using TR = TailRaw<ED, KB1>;
  const uint16_t* emb = (const uint16_t*)a.emb;
#pragma unroll
  for (int kb = 0; kb < TR::KE; ++kb) x[kb] = *(const u32x4*)(emb + (size_t)c.q * ED + 16 * kb + 8 * g);
  const int n4 = 4 * a.M;
#pragma unroll
  for (int t = 0; t < TR::KT; ++t) {
    const int k2 = 16 * t + 8 * g;
    const float* row = a.snap + (size_t)c.e * snap_stride(a.M) + (k2 < n4 ? k2 : n4 - 1);
    raw.t[t][0] = *(const float4*)row;
    raw.t[t][1] = *(const float4*)(row + 4);
  }
}
template <int ED, int KB1>
__device__ __forceinline__ void gather_finish(const RouteArgs& a, const RowCtx& c, int g, u32x4 (&x)[KB1],
                                              const TailRaw<ED, KB1>& raw) {
  using TR = TailRaw<ED, KB1>;
  const int n4 = 4 * a.M;
  const float fb = (float)c.budget * a.inv_bud;
#pragma unroll
  for (int t = 0; t < TR::KT; ++t) {
    const int k2 = 16 * t + 8 * g;
    const float4 lo = raw.t[t][0], hi = raw.t[t][1];
    const float v[8] = {lo.x, lo.y, lo.z, lo.w, hi.x, hi.y, hi.z, hi.w};
    float f[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int kk = k2 + i;
      f[i] = kk < n4 ? v[i] : (kk == n4 ? fb : 0.f);
    }
    u32x4 r;
    r.x = pack2(f[0], f[1]);
    r.y = pack2(f[2], f[3]);
    r.z = pack2(f[4], f[5]);
    r.w = pack2(f[6], f[7]);
    x[TR::KE + t] = r;
  }
}

// Philox4x32-10 block (Salmon, Moraes, Dror, Shaw, SC 2011): ten rounds of
// two 32x32 -> 64-bit products by the round multipliers, whose high halves are
// xored with the other two counter words and the key; the key advances by the
// Weyl constants after every round.
__device__ __forceinline__ uint4 philox10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    // one 32x32 -> 64-bit product each (a single v_mad_u64_u32)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c.w ^ k1,
                   (uint32_t)p0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// Exponential variate E = -ln U of a 32-bit word, U = (top 23 bits + 1/2)
// 2^-23 (exact in fp32). Above U = 15/16, 1 - U = d is exact and -ln(1 - d)
// is summed as d + d^2/2 + ... + d^7/7 (the rest is below 2^-24 d), so E keeps
// its relative precision however close U is to 1.
__device__ __forceinline__ float expo_of(uint32_t w) {
  const uint32_t k = w >> 9;
  const float u = ((float)k + 0.5f) * (1.0f / 8388608.0f);
  const float d = ((float)(8388608u - k) - 0.5f) * (1.0f / 8388608.0f);
  const float series =
      d * (1.f + d * (0.5f + d * (1.f / 3.f + d * (0.25f + d * (0.2f + d * (1.f / 6.f + d * (1.f / 7.f)))))));
  return d < 0.0625f ? series : -__logf(u);
}

// RL-rollout outputs of one row from its logits (lane pair n, n + 32 holds
// the row's actions 32 T + 8 (v / 4) + 4 g + v % 4): pi is the softmax of
// the logits over the valid actions, shifted by their largest logit `zmax`
// (action `amax`, -1 when none is valid); the action is the Gumbel-max draw
// (or `amax` when greedy), its log-probability z_a - logsumexp, the entropy
// logsumexp - sum pi z, and the value head's row A. The Gumbel-max draw
// argmax z_a - ln(E_a), E_a = -ln U_a, is taken as the equivalent argmax of
// exp(z_a - zmax) / E_a (one logarithm per action instead of two).
template <int AT>
__device__ __forceinline__ void rl_outputs(const RouteArgs& a, const RowCtx& c,
                                           const f32x16 (&acc)[AT], int g, float zmax, int amax) {
  const bool sample = a.greedy == 0;
  uint32_t id = 0;
  if (sample) {
    const int32_t rr = c.live ? c.r : a.n_total - 1;
    id = (uint32_t)(a.ms[(size_t)c.e * a.M].next_id + (rr - a.offsets[c.e]));
  }
  float s = 0.f, sz = 0.f, val = 0.f, bs = 0.f, bz = 0.f;
  int bsa = -1;
#pragma unroll
  for (int T = 0; T < AT; ++T) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int a0 = 32 * T + 8 * j + 4 * g;   // this lane's 4 consecutive actions: one Philox block
      uint4 w = make_uint4(0, 0, 0, 0);
      if (sample && a0 < a.A) w = philox10(make_uint4(id, (uint32_t)c.e, (uint32_t)(a0 >> 2), 0u), a.seed_lo, a.seed_hi);
      const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int act = a0 + i;
        const float z = acc[T][4 * j + i];
        if (act == a.A) val = z;
        if (act < a.A && ((c.amask >> act) & 1ull)) {
          const float ex = __expf(z - zmax);
          s += ex;
          sz += ex * z;
          const float sc = sample ? __fdividef(ex, expo_of(wv[i])) : z;
          if (bsa < 0 || sc > bs) { bs = sc; bsa = act; bz = z; }   // actions ascend: ties keep the lowest
        }
      }
    }
  }
  s += __shfl_xor(s, 32, 64);
  sz += __shfl_xor(sz, 32, 64);
  val += __shfl_xor(val, 32, 64);                  // one lane of the pair holds row A
  const float obs = __shfl_xor(bs, 32, 64), obz = __shfl_xor(bz, 32, 64);
  const int obsa = __shfl_xor(bsa, 32, 64);
  if (obsa >= 0 && (bsa < 0 || obs > bs || (obs == bs && obsa < bsa))) { bs = obs; bsa = obsa; bz = obz; }
  if (!c.live || g != 0) return;
  const bool any = amax >= 0 && !c.bad;
  const float lse = any ? zmax + __logf(s) : 0.f;
  a.actions[c.r] = any ? bsa : -1;
  if (c.bad) atomicOr(a.err, c.bad);
  if (a.logp) a.logp[c.r] = any ? bz - lse : 0.f;
  if (a.entropy) a.entropy[c.r] = any ? lse - sz / s : 0.f;
  if (a.value) a.value[c.r] = c.bad ? 0.f : val;
}

// Masked argmax over the lane pair (n, n + 32), logits store, action store
// (or the RL-rollout outputs). RL: 0 = greedy route only, 1 = RL outputs
// only, 2 = either, chosen by a.rl at run time.
template <int AT, int RL = 2>
__device__ __forceinline__ void epilogue(const RouteArgs& a, const RowCtx& c, f32x16 (&acc)[AT],
                                         const float* bias, int g) {
  float best = 0.f;
  int ba = -1;
#pragma unroll
  for (int T = 0; T < AT; ++T) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int act = 32 * T + 8 * (v >> 2) + 4 * g + (v & 3);
      const float z = bias ? acc[T][v] + bias[(T * 2 + g) * 16 + v] : acc[T][v];
      acc[T][v] = z;
      if (act < a.A && ((c.amask >> act) & 1ull)) {
        if (ba < 0 || z > best) { best = z; ba = act; }
      }
    }
  }
  const float ob = __shfl_xor(best, 32, 64);
  const int oa = __shfl_xor(ba, 32, 64);
  if (oa >= 0 && (ba < 0 || ob > best || (ob == best && oa < ba))) { best = ob; ba = oa; }
  if (RL == 1 || (RL == 2 && a.rl)) {
    rl_outputs<AT>(a, c, acc, g, best, ba);
  } else if (c.live && g == 0) {
    a.actions[c.r] = c.bad ? -1 : ba;
    if (c.bad) atomicOr(a.err, c.bad);
  }
  if (!c.live) return;
  if (a.logits) {
    float* out = a.logits + (size_t)c.r * a.A;
#pragma unroll
    for (int T = 0; T < AT; ++T) {
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int act = 32 * T + 8 * (v >> 2) + 4 * g + (v & 3);
        if (act < a.A) out[act] = c.bad ? 0.f : acc[T][v];
      }
    }
  }
}

// bias + ReLU + bf16 rounding of one accumulator tile into two B fragments.
__device__ __forceinline__ void tile_to_frags(const f32x16& acc, const float* bias, int T, int g,
                                              u32x4& f0, u32x4& f1) {
  float h[16];
#pragma unroll
  for (int v = 0; v < 16; ++v) h[v] = acc[v] + bias[(T * 2 + g) * 16 + v];
  f0.x = relu_pack2(h[0], h[1]);   f0.y = relu_pack2(h[2], h[3]);
  f0.z = relu_pack2(h[4], h[5]);   f0.w = relu_pack2(h[6], h[7]);
  f1.x = relu_pack2(h[8], h[9]);   f1.y = relu_pack2(h[10], h[11]);
  f1.z = relu_pack2(h[12], h[13]); f1.w = relu_pack2(h[14], h[15]);
}

// ReLU + bf16 rounding of one accumulator tile (bias already included).
__device__ __forceinline__ void relu_to_frags(const f32x16& acc, u32x4& f0, u32x4& f1) {
  f0.x = relu_pack2(acc[0], acc[1]);   f0.y = relu_pack2(acc[2], acc[3]);
  f0.z = relu_pack2(acc[4], acc[5]);   f0.w = relu_pack2(acc[6], acc[7]);
  f1.x = relu_pack2(acc[8], acc[9]);   f1.y = relu_pack2(acc[10], acc[11]);
  f1.z = relu_pack2(acc[12], acc[13]); f1.w = relu_pack2(acc[14], acc[15]);
}

template <int H, int NL, int AT>
__global__ __launch_bounds__(256) void route_bf16(RouteArgs a_in) {
  // chain pools: the tick's row count is on the device
  RouteArgs a = a_in;
  if (a_in.n_total_dev) a.n_total = min(*a_in.n_total_dev, a_in.n_total);   // the caller's buffers bound it
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, g = lane >> 5;
  const int32_t row0 = (int32_t)(blockIdx.x * 4 + wave) * 32;
  if (row0 >= a.n_total) return;
  const RowCtx c = row_setup(a, row0, row0 + n);
  constexpr int TH = H / 32;        // hidden tiles
  constexpr int KH = H / 16;        // K blocks over a hidden layer
  const u32x4* W1 = (const u32x4*)a.W[0];
  f32x16 acc[TH];
#pragma unroll
  for (int T = 0; T < TH; ++T) acc[T] = f32x16{};
  for (int kb = 0; kb < a.k1; ++kb) {
    const u32x4 xb = gather_bf16(a, c, kb, g);
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

// ---------------------------------------------------------------------------
// fp32 policies on v_mfma_f32_16x16x4_f32, one wave per 16 rows (a light
// fp32 tick, ~16 K requests, still gives every SIMD a wave).
//
// Transposed form Y^T = W X^T: lane l serves row n = l % 16 of the wave's
// rows and K group q = l / 16. An output tile's accumulator holds features
// 16 T + 4 q + r (r = 0..3) of the lane's row: exactly the B operand of the
// next layer's K step (T, r), whose weight columns are permuted to match at
// pool creation, so activations never leave registers. Weights are packed so
// that one 16-byte load per lane covers four consecutive K steps; the hidden
// layers' loads run D steps ahead of their MFMAs.
// ---------------------------------------------------------------------------

// Masked argmax over the four lanes of a row (q = 0..3), action and logits
// stores, or the RL-rollout outputs; lane (n, q) holds actions 16 T + 4 q + r.
// Same rules as the 32-row epilogue: lowest action on exact ties, Philox block
// (id, env, action / 4) per four consecutive actions.
template <int AT>
__device__ __forceinline__ void epilogue16(const RouteArgs& a, const RowCtx& c, const f32x4 (&acc)[AT], int q) {
  float best = 0.f;
  int ba = -1;
#pragma unroll
  for (int T = 0; T < AT; ++T) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int act = 16 * T + 4 * q + r;
      const float z = acc[T][r];
      if (act < a.A && ((c.amask >> act) & 1ull)) {
        if (ba < 0 || z > best) { best = z; ba = act; }
      }
    }
  }
#pragma unroll
  for (int off = 16; off <= 32; off *= 2) {
    const float ob = __shfl_xor(best, off, 64);
    const int oa = __shfl_xor(ba, off, 64);
    if (oa >= 0 && (ba < 0 || ob > best || (ob == best && oa < ba))) { best = ob; ba = oa; }
  }
  if (a.rl) {
    const bool sample = a.greedy == 0;
    uint32_t id = 0;
    if (sample) {
      const int32_t rr = c.live ? c.r : a.n_total - 1;
      id = (uint32_t)(a.ms[(size_t)c.e * a.M].next_id + (rr - a.offsets[c.e]));
    }
    float sm = 0.f, sz = 0.f, val = 0.f, bs = 0.f, bz = 0.f;
    int bsa = -1;
#pragma unroll
    for (int T = 0; T < AT; ++T) {
      const int a0 = 16 * T + 4 * q;   // this lane's 4 consecutive actions: one Philox block
      uint4 w = make_uint4(0, 0, 0, 0);
      if (sample && a0 < a.A) w = philox10(make_uint4(id, (uint32_t)c.e, (uint32_t)(a0 >> 2), 0u), a.seed_lo, a.seed_hi);
      const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int act = a0 + i;
        const float z = acc[T][i];
        if (act == a.A) val = z;
        if (act < a.A && ((c.amask >> act) & 1ull)) {
          const float ex = __expf(z - best);
          sm += ex;
          sz += ex * z;
          const float sc = sample ? __fdividef(ex, expo_of(wv[i])) : z;
          if (bsa < 0 || sc > bs) { bs = sc; bsa = act; bz = z; }   // actions ascend: ties keep the lowest
        }
      }
    }
#pragma unroll
    for (int off = 16; off <= 32; off *= 2) {
      sm += __shfl_xor(sm, off, 64);
      sz += __shfl_xor(sz, off, 64);
      val += __shfl_xor(val, off, 64);             // one lane of the row holds row A
      const float obs = __shfl_xor(bs, off, 64), obz = __shfl_xor(bz, off, 64);
      const int obsa = __shfl_xor(bsa, off, 64);
      if (obsa >= 0 && (bsa < 0 || obs > bs || (obs == bs && obsa < bsa))) { bs = obs; bsa = obsa; bz = obz; }
    }
    if (c.live && q == 0) {
      const bool any = ba >= 0 && !c.bad;
      const float lse = any ? best + __logf(sm) : 0.f;
      a.actions[c.r] = any ? bsa : -1;
      if (c.bad) atomicOr(a.err, c.bad);
      if (a.logp) a.logp[c.r] = any ? bz - lse : 0.f;
      if (a.entropy) a.entropy[c.r] = any ? lse - sz / sm : 0.f;
      if (a.value) a.value[c.r] = c.bad ? 0.f : val;
    }
  } else if (c.live && q == 0) {
    a.actions[c.r] = c.bad ? -1 : ba;
    if (c.bad) atomicOr(a.err, c.bad);
  }
  if (!c.live) return;
  if (a.logits) {
    float* out = a.logits + (size_t)c.r * a.A;
#pragma unroll
    for (int T = 0; T < AT; ++T) {
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int act = 16 * T + 4 * q + r;
        if (act < a.A) out[act] = c.bad ? 0.f : acc[T][r];
      }
    }
  }
}

// One hidden-input layer: out[To] = bias + W h over K = 4 KG steps, the
// weights of step group (To, g) at W[(To KG + g) 64 + lane] (4 floats, one
// per K step of the group). With one wave per SIMD the MFMAs are ordered so
// that consecutive ones never share an accumulator: four output tiles at a
// time (weights of D groups in flight), or, for fewer than four tiles, each
// tile's K steps split over four partial sums added at the end.
template <int TO, int KG, int D>
__device__ __forceinline__ void layer16(const f32x4* W, const float* bias, const f32x4 (&h)[KG], int lane,
                                        int q, f32x4 (&out)[TO]) {
  if constexpr (TO % 4 == 0) {
    constexpr int N = (TO / 4) * KG;   // (tile quad, group) steps
    constexpr int DD = D < N ? D : N;
    f32x4 wr[DD][4];
    auto load = [&](int s, f32x4 (&w)[4]) {
      const int T4 = s / KG, g = s % KG;
#pragma unroll
      for (int t = 0; t < 4; ++t) w[t] = W[((4 * T4 + t) * KG + g) * 64 + lane];
    };
#pragma unroll
    for (int s = 0; s < DD; ++s) load(s, wr[s]);
#pragma unroll
    for (int T4 = 0; T4 < TO / 4; ++T4) {
      f32x4 acc[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) acc[t] = *(const f32x4*)(bias + ((4 * T4 + t) * 4 + q) * 4);
#pragma unroll
      for (int g = 0; g < KG; ++g) {
        const int st = T4 * KG + g;
        f32x4 w[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) w[t] = wr[st % DD][t];
        if (st + DD < N) load(st + DD, wr[st % DD]);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma16_f32(w[t].x, h[g].x, acc[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma16_f32(w[t].y, h[g].y, acc[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma16_f32(w[t].z, h[g].z, acc[t]);
#pragma unroll
        for (int t = 0; t < 4; ++t) acc[t] = mfma16_f32(w[t].w, h[g].w, acc[t]);
      }
#pragma unroll
      for (int t = 0; t < 4; ++t) out[4 * T4 + t] = acc[t];
    }
  } else {
    constexpr int N = TO * KG;
    constexpr int DD = 4 * D < N ? 4 * D : N;
    f32x4 wr[DD];
#pragma unroll
    for (int t = 0; t < DD; ++t) wr[t] = W[t * 64 + lane];
#pragma unroll
    for (int To = 0; To < TO; ++To) {
      f32x4 p[4];
      p[0] = *(const f32x4*)(bias + (To * 4 + q) * 4);
      p[1] = p[2] = p[3] = f32x4{};
#pragma unroll
      for (int g = 0; g < KG; ++g) {
        const int t = To * KG + g;
        const f32x4 w = wr[t % DD];
        if (t + DD < N) wr[t % DD] = W[(t + DD) * 64 + lane];
        p[0] = mfma16_f32(w.x, h[g].x, p[0]);
        p[1] = mfma16_f32(w.y, h[g].y, p[1]);
        p[2] = mfma16_f32(w.z, h[g].z, p[2]);
        p[3] = mfma16_f32(w.w, h[g].w, p[3]);
      }
      out[To] = (p[0] + p[1]) + (p[2] + p[3]);
    }
  }
}

template <int H, int NL, int AT>
__global__ __launch_bounds__(256) void route_f32(RouteArgs a_in) {
  // chain pools: the tick's row count is on the device
  RouteArgs a = a_in;
  if (a_in.n_total_dev) a.n_total = min(*a_in.n_total_dev, a_in.n_total);   // the caller's buffers bound it
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 15, q = lane >> 4;
  const int32_t row0 = (int32_t)(blockIdx.x * 4 + wave) * 16;
  if (row0 >= a.n_total) return;
  const int32_t rl = row0 + 15 < a.n_total ? row0 + 15 : a.n_total - 1;
  const int32_t rows[1] = {row0 + n};
  const int32_t rsel[1] = {rows[0] < a.n_total ? rows[0] : a.n_total - 1};
  int32_t envs[1];
  find_envs<1>(a, row0, rl, rsel, envs);
  const RowCtx c = row_setup_env(a, rows[0], envs[0]);
  constexpr int TH = H / 16;   // hidden output tiles
  constexpr int KGH = H / 16;  // K step groups over a hidden layer (4 steps of 4 features)
  const f32x4* W1 = (const f32x4*)a.W[0];
  const float* emb = (const float*)a.emb + (size_t)c.q * a.embed_dim;
  // layer 1: K step s, lane group q carries feature 4 s + q; four steps per group
  const int KG1 = (a.k1 + 3) / 4;
  f32x4 h1[TH];
#pragma unroll
  for (int T = 0; T < TH; ++T) h1[T] = *(const f32x4*)(a.bias[0] + (T * 4 + q) * 4);
  auto feats = [&](int g) {
    f32x4 x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = 16 * g + 4 * j + q;
      x[j] = k < a.embed_dim ? emb[k] : tail_feature(a, c, k);
    }
    return x;
  };
  f32x4 x = feats(0);
  f32x4 wn[TH];
#pragma unroll
  for (int T = 0; T < TH; ++T) wn[T] = W1[(T * KG1) * 64 + lane];
  for (int g = 0; g < KG1; ++g) {
    f32x4 wc[TH];
#pragma unroll
    for (int T = 0; T < TH; ++T) wc[T] = wn[T];
    const f32x4 xc = x;
    if (g + 1 < KG1) {
      x = feats(g + 1);
#pragma unroll
      for (int T = 0; T < TH; ++T) wn[T] = W1[(T * KG1 + g + 1) * 64 + lane];
    }
    // K step by K step across the output tiles: consecutive MFMAs never
    // share an accumulator
#pragma unroll
    for (int T = 0; T < TH; ++T) h1[T] = mfma16_f32(wc[T].x, xc.x, h1[T]);
#pragma unroll
    for (int T = 0; T < TH; ++T) h1[T] = mfma16_f32(wc[T].y, xc.y, h1[T]);
#pragma unroll
    for (int T = 0; T < TH; ++T) h1[T] = mfma16_f32(wc[T].z, xc.z, h1[T]);
#pragma unroll
    for (int T = 0; T < TH; ++T) h1[T] = mfma16_f32(wc[T].w, xc.w, h1[T]);
  }
#pragma unroll
  for (int T = 0; T < TH; ++T)
#pragma unroll
    for (int r = 0; r < 4; ++r) h1[T][r] = relu(h1[T][r]);
  f32x4 out[AT];
  if constexpr (NL == 2) {
    layer16<AT, KGH, 2>((const f32x4*)a.W[1], a.bias[1], h1, lane, q, out);
  } else {
    f32x4 h2[TH];
    layer16<TH, KGH, 2>((const f32x4*)a.W[1], a.bias[1], h1, lane, q, h2);
#pragma unroll
    for (int T = 0; T < TH; ++T)
#pragma unroll
      for (int r = 0; r < 4; ++r) h2[T][r] = relu(h2[T][r]);
    layer16<AT, KGH, 2>((const f32x4*)a.W[2], a.bias[2], h2, lane, q, out);
  }
  epilogue16<AT>(a, c, out, q);
}

// TQ output tiles [To0, To0 + TQ) of a layer over its hidden input, read from
// LDS (`hs`: tile g's 16-byte words at hs[g 64 + lane]) while the weights
// (W[(To KG + g) 64 + lane], 4 floats) come through the caches D groups
// ahead. Consecutive MFMAs use different accumulators: the tiles' own chains
// when there are four or more, else four partial sums per tile.
template <int TQ, int KG, int D>
__device__ __forceinline__ void layer16_lds(const f32x4* W, const float* bias, const f32x4* hs, int To0,
                                            int lane, int q, f32x4 (&out)[TQ]) {
  constexpr int NP = TQ >= 4 ? 1 : 4;
  constexpr int DD = D < KG ? D : KG;
  f32x4 wr[DD][TQ];
#pragma unroll
  for (int g = 0; g < DD; ++g)
#pragma unroll
    for (int t = 0; t < TQ; ++t) wr[g][t] = W[((To0 + t) * KG + g) * 64 + lane];
  f32x4 acc[TQ][NP];
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
    acc[t][0] = *(const f32x4*)(bias + ((To0 + t) * 4 + q) * 4);
#pragma unroll
    for (int i = 1; i < NP; ++i) acc[t][i] = f32x4{};
  }
  f32x4 bn = hs[lane];
#pragma unroll
  for (int g = 0; g < KG; ++g) {
    const f32x4 b = bn;
    if (g + 1 < KG) bn = hs[(g + 1) * 64 + lane];
    f32x4 w[TQ];
#pragma unroll
    for (int t = 0; t < TQ; ++t) w[t] = wr[g % DD][t];
    if (g + DD < KG) {
#pragma unroll
      for (int t = 0; t < TQ; ++t) wr[g % DD][t] = W[((To0 + t) * KG + g + DD) * 64 + lane];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < TQ; ++t) acc[t][j % NP] = mfma16_f32(w[t][j], b[j], acc[t][j % NP]);
  }
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
    f32x4 r = acc[t][0];
#pragma unroll
    for (int i = 1; i < NP; ++i) r += acc[t][i];
    out[t] = r;
  }
}

// fp32 policies with hidden widths in whole tile quads, feature-split: one
// block of 4 waves per 16-row tile, wave w computing output tiles
// [w TH/4, (w + 1) TH/4) of each hidden layer; the block exchanges a layer's
// activations through LDS (one 16-row x H buffer, h1 and then h2), and wave 0
// computes the output layer and the epilogue. Each wave does about a quarter
// of a tile's MFMAs, so four waves share each SIMD and hide each other's
// latencies, and a tick slightly above a multiple of the machine's SIMDs
// adds quarter tiles rather than whole ones.
template <int H, int NL, int AT>
__global__ __launch_bounds__(256) void route_f32s(RouteArgs a_in) {
  // chain pools: the tick's row count is on the device
  RouteArgs a = a_in;
  if (a_in.n_total_dev) a.n_total = min(*a_in.n_total_dev, a_in.n_total);   // the caller's buffers bound it
  constexpr int TH = H / 16, TQ = TH / 4, KGH = H / 16;
  static_assert(TH % 4 == 0, "hidden tiles split four ways");
  __shared__ f32x4 hs[TH * 64];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int n = lane & 15, q = lane >> 4;
  const int32_t row0 = (int32_t)blockIdx.x * 16;
  if (row0 >= a.n_total) return;   // the whole block (chain pools' bound launch)
  const int32_t rl = row0 + 15 < a.n_total ? row0 + 15 : a.n_total - 1;
  const int32_t rows[1] = {row0 + n};
  const int32_t rsel[1] = {rows[0] < a.n_total ? rows[0] : a.n_total - 1};
  int32_t envs[1];
  find_envs<1>(a, row0, rl, rsel, envs);
  const RowCtx c = row_setup_env(a, rows[0], envs[0]);
  const int T0 = wave * TQ;
  // layer 1 (this wave's tiles): K step s, lane group q carries feature 4 s + q
  const f32x4* W1 = (const f32x4*)a.W[0];
  const float* emb = (const float*)a.emb + (size_t)c.q * a.embed_dim;
  const int KG1 = (a.k1 + 3) / 4;
  f32x4 h1[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) h1[t] = *(const f32x4*)(a.bias[0] + ((T0 + t) * 4 + q) * 4);
  auto feats = [&](int g) {
    f32x4 x;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int k = 16 * g + 4 * j + q;
      x[j] = k < a.embed_dim ? emb[k] : tail_feature(a, c, k);
    }
    return x;
  };
  f32x4 x = feats(0);
  f32x4 wn[TQ];
#pragma unroll
  for (int t = 0; t < TQ; ++t) wn[t] = W1[((T0 + t) * KG1) * 64 + lane];
  for (int g = 0; g < KG1; ++g) {
    f32x4 wc[TQ];
#pragma unroll
    for (int t = 0; t < TQ; ++t) wc[t] = wn[t];
    const f32x4 xc = x;
    if (g + 1 < KG1) {
      x = feats(g + 1);
#pragma unroll
      for (int t = 0; t < TQ; ++t) wn[t] = W1[((T0 + t) * KG1 + g + 1) * 64 + lane];
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int t = 0; t < TQ; ++t) h1[t] = mfma16_f32(wc[t][j], xc[j], h1[t]);
  }
#pragma unroll
  for (int t = 0; t < TQ; ++t) {
#pragma unroll
    for (int r = 0; r < 4; ++r) h1[t][r] = relu(h1[t][r]);
    hs[(T0 + t) * 64 + lane] = h1[t];
  }
  __syncthreads();
  if constexpr (NL == 3) {
    f32x4 h2[TQ];
    layer16_lds<TQ, KGH, 2>((const f32x4*)a.W[1], a.bias[1], hs, T0, lane, q, h2);
    __syncthreads();   // every wave is done reading h1
#pragma unroll
    for (int t = 0; t < TQ; ++t) {
#pragma unroll
      for (int r = 0; r < 4; ++r) h2[t][r] = relu(h2[t][r]);
      hs[(T0 + t) * 64 + lane] = h2[t];
    }
    __syncthreads();
  }
  if (wave != 0) return;
  f32x4 out[AT];
  layer16_lds<AT, KGH, 2>((const f32x4*)a.W[NL - 1], a.bias[NL - 1], hs, 0, lane, q, out);
  epilogue16<AT>(a, c, out, q);
}

// ---------------------------------------------------------------------------
// Persistent variant for policies whose deeper layers fit in LDS.
//
// Each block (NW waves) copies the packed weights of layers >= 2 (and of
// layer 1 when it also fits) into LDS once, then its waves take turns over
// the block's share of wave tiles. A wave tile is NR 32-row MFMA column tiles,
// so every weight fragment read feeds NR MFMAs. Layer-1 outputs are produced
// one 32-feature tile at a time and rounded to bf16 fragments right away.
// ---------------------------------------------------------------------------

// Copies n 16-byte words from global memory to LDS with `nthreads` threads,
// batches of 8 loads in flight per thread.
template <int N, int NTHREADS>
__device__ __forceinline__ void copy_to_lds(u32x4* dst, const u32x4* src) {
  constexpr int PER = (N + NTHREADS - 1) / NTHREADS;
  constexpr int B = 8;
#pragma unroll
  for (int b0 = 0; b0 < PER; b0 += B) {
    u32x4 v[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int i = (b0 + j) * NTHREADS + (int)threadIdx.x;
      if (b0 + j < PER && i < N) v[j] = src[i];
    }
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int i = (b0 + j) * NTHREADS + (int)threadIdx.x;
      if (b0 + j < PER && i < N) dst[i] = v[j];
    }
  }
}

// Wave tiles (32 NR rows each) of block b in a persistent grid of G blocks:
// the contiguous range [first, end) of an equal split of all n_units (the
// shares differ by at most one tile). A row count just above a multiple of
// the grid's capacity then adds one tile to a few blocks instead of a whole
// extra round of tiles to one block.
struct UnitRange {
  int32_t first, end;
};
__device__ __forceinline__ UnitRange block_units(int32_t n_units) {
  UnitRange u;
  u.first = (int32_t)(((int64_t)blockIdx.x * n_units) / gridDim.x);
  u.end = (int32_t)(((int64_t)(blockIdx.x + 1) * n_units) / gridDim.x);
  return u;
}

template <int H, int NL, int AT, int KB1, bool W1L, int NW, int ED, int NR, int RL, int W1PF, bool PIPE>
__global__ __launch_bounds__(NW * 64, 1) void route_bf16_lds(RouteArgs a_in) {
  // chain pools: the tick's row count is on the device
  RouteArgs a = a_in;
  if (a_in.n_total_dev) a.n_total = min(*a_in.n_total_dev, a_in.n_total);   // the caller's buffers bound it
  constexpr int TH = H / 32;
  constexpr int KH = H / 16;
  constexpr int N_W1 = TH * KB1 * 64;
  constexpr int N_W2 = (NL == 3 ? TH : AT) * KH * 64;
  constexpr int N_W3 = NL == 3 ? AT * KH * 64 : 0;
  constexpr int N_LDS = (W1L ? N_W1 : 0) + N_W2 + N_W3;
  // biases in accumulator-register order: [tile][g][16] floats per layer
  constexpr int NB0 = TH * 32, NB1 = (NL == 3 ? TH : AT) * 32, NB2 = NL == 3 ? AT * 32 : 0;
  constexpr int WROWS = 32 * NR;            // rows per wave tile
  __shared__ u32x4 lds[N_LDS];
  __shared__ float lbias[NB0 + NB1 + NB2];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform loop control
  const int n = lane & 31, g = lane >> 5;
  const UnitRange ur = block_units((a.n_total + WROWS - 1) / WROWS);
  // Wave tile u is set up in two steps: its first loads (the CSR window and
  // the rows' q_idx and budget), then, once they have arrived, the env
  // lookup, the env's snapshot row and the embedding rows (row contexts and
  // layer-1 B fragments).
  struct First {
    EnvWindow w;
    int32_t q[NR], bud[NR];
  };
  auto first_loads = [&](int32_t u) {
    First f;
    const int32_t r0 = u * WROWS;
    f.w = env_window(a, r0);
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      const int32_t r = r0 + 32 * j + n;
      const int32_t rr = r < a.n_total ? r : a.n_total - 1;
      f.q[j] = a.q_idx[rr];
      f.bud[j] = a.budget[rr];
    }
    return f;
  };
  auto setup = [&](int32_t u, const First& f, RowCtx (&c)[NR], u32x4 (&x)[NR][KB1], int gg) {
    const int32_t r0 = u * WROWS;
    const int32_t rlast = (r0 + WROWS - 1 < a.n_total ? r0 + WROWS - 1 : a.n_total - 1);
    int32_t rows[NR], envs[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) rows[j] = r0 + 32 * j + n;
    find_envs_in<NR>(a, f.w, r0, rlast, rows, envs);
    ValidRaw vr[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      c[j] = row_ctx_from(a, rows[j], envs[j], f.q[j], f.bud[j]);
      vr[j] = load_valid(a, envs[j]);
    }
    TailRaw<ED, KB1> raw[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) gather_issue<ED, KB1>(a, c[j], gg, x[j], raw[j]);
    // the masks wait only for their own words: the embedding and snapshot
    // loads issued after them stay in flight
#pragma unroll
    for (int j = 0; j < NR; ++j) c[j].amask = mask_of(a, vr[j]);
#pragma unroll
    for (int j = 0; j < NR; ++j) gather_finish<ED, KB1>(a, c[j], gg, x[j], raw[j]);
  };
  // PIPE: the first wave tile is set up (first loads, then its gather)
  // while the block copies the weights into LDS, before the barrier, and each
  // later tile at the end of the previous iteration, so the loop starts with
  // layer 1 (its inputs are loop-carried: this pays only where the registers
  // are not all taken).
  int32_t u = ur.first + wave;
  RowCtx c[NR];
  u32x4 x[NR][KB1];
  First f0;
  if (PIPE && u < ur.end) f0 = first_loads(u);
  if constexpr (W1L) copy_to_lds<N_W1, NW * 64>(lds, (const u32x4*)a.W[0]);
  copy_to_lds<N_W2, NW * 64>(lds + (W1L ? N_W1 : 0), (const u32x4*)a.W[1]);
  if constexpr (NL == 3) copy_to_lds<N_W3, NW * 64>(lds + (W1L ? N_W1 : 0) + N_W2, (const u32x4*)a.W[2]);
  for (int i = threadIdx.x; i < NB0 + NB1 + NB2; i += NW * 64)
    lbias[i] = i < NB0 ? a.bias[0][i] : (i < NB0 + NB1 ? a.bias[1][i - NB0] : a.bias[2][i - NB0 - NB1]);
  if constexpr (PIPE) {
    if (u < ur.end) setup(u, f0, c, x, g);
  }
  __syncthreads();
  if (u >= ur.end) return;
  const float* lb0 = lbias;
  const float* lb1 = lbias + NB0;
  const float* lb2 = lbias + NB0 + NB1;
  const u32x4* w1 = W1L ? (const u32x4*)lds : (const u32x4*)a.W[0];
  const u32x4* w2 = lds + (W1L ? N_W1 : 0);
  const u32x4* w3 = w2 + N_W2;

  for (;;) {
    // Keeps loop-invariant loads (biases, weights) inside the loop: hoisted
    // out of it they would stay live in registers for the whole kernel.
    asm volatile("" ::: "memory");
    // Per-iteration copies of the lane index: every fragment address derived
    // from them is recomputed inside the iteration instead of being hoisted
    // (and kept live) across the whole loop.
    int ln = lane, gg = g;
    asm volatile("" : "+v"(ln), "+v"(gg));
    if constexpr (!PIPE) setup(u, first_loads(u), c, x, gg);

    u32x4 h[NR][NL == 3 ? KH : 1];
    // two-layer policies: the output layer consumes each layer-1 output tile
    // as soon as it is rounded (its two K steps), so the hidden layer is
    // never held whole
    f32x16 o[NR][AT];
    if constexpr (NL == 2) {
#pragma unroll
      for (int T = 0; T < AT; ++T) {
        o[0][T] = *(const f32x16*)(lb1 + (T * 2 + gg) * 16);
#pragma unroll
        for (int j = 1; j < NR; ++j) o[j][T] = o[0][T];
      }
    }
    // layer-1 fragments: W1PF of the next output tile's K steps are loaded
    // while the current tile's MFMAs run (the rest just before they are used)
    u32x4 wk[KB1], wn[KB1];
#pragma unroll
    for (int kb = 0; kb < KB1; ++kb) wn[kb] = w1[kb * 64 + ln];
#pragma unroll
    for (int cc = 0; cc < TH; ++cc) {
#pragma unroll
      for (int kb = 0; kb < KB1; ++kb) wk[kb] = kb < W1PF || cc == 0 ? wn[kb] : w1[(cc * KB1 + kb) * 64 + ln];
      if (cc + 1 < TH) {
#pragma unroll
        for (int kb = 0; kb < W1PF; ++kb) wn[kb] = w1[((cc + 1) * KB1 + kb) * 64 + ln];
      }
      f32x16 p[NR];
      p[0] = *(const f32x16*)(lb0 + (cc * 2 + gg) * 16);
#pragma unroll
      for (int j = 1; j < NR; ++j) p[j] = p[0];
#pragma unroll
      for (int kb = 0; kb < KB1; ++kb) {
#pragma unroll
        for (int j = 0; j < NR; ++j) p[j] = mfma_bf16(wk[kb], x[j][kb], p[j]);
      }
      if constexpr (NL == 2) {
        u32x4 f[NR][2];
#pragma unroll
        for (int j = 0; j < NR; ++j) relu_to_frags(p[j], f[j][0], f[j][1]);
#pragma unroll
        for (int T = 0; T < AT; ++T) {
          const u32x4 wa = w2[(T * KH + 2 * cc) * 64 + ln];
          const u32x4 wb = w2[(T * KH + 2 * cc + 1) * 64 + ln];
#pragma unroll
          for (int j = 0; j < NR; ++j) {
            o[j][T] = mfma_bf16(wa, f[j][0], o[j][T]);
            o[j][T] = mfma_bf16(wb, f[j][1], o[j][T]);
          }
        }
      } else {
#pragma unroll
        for (int j = 0; j < NR; ++j) relu_to_frags(p[j], h[j][2 * cc], h[j][2 * cc + 1]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    if constexpr (NL == 3) {
#pragma unroll
      for (int T = 0; T < AT; ++T) {
        o[0][T] = *(const f32x16*)(lb2 + (T * 2 + gg) * 16);
#pragma unroll
        for (int j = 1; j < NR; ++j) o[j][T] = o[0][T];
      }
#pragma unroll
      for (int cc = 0; cc < TH; ++cc) {
        f32x16 p[NR];
        p[0] = *(const f32x16*)(lb1 + (cc * 2 + gg) * 16);
#pragma unroll
        for (int j = 1; j < NR; ++j) p[j] = p[0];
        // LDS fragments two K steps ahead of the MFMAs that use them
        u32x4 w_0 = w2[(cc * KH + 0) * 64 + ln];
        u32x4 w_1 = w2[(cc * KH + 1) * 64 + ln];
        // the wave raises its issue priority for the chain of MFMAs, so that
        // the other wave of its SIMD runs its ReLU, packing and loads in the
        // chain's shadow instead of taking turns on the matrix pipe
        if constexpr (!PIPE && NR == 2) __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int kb = 0; kb < KH; ++kb) {
          const u32x4 w_2 = w2[(cc * KH + (kb + 2 < KH ? kb + 2 : KH - 1)) * 64 + ln];
#pragma unroll
          for (int j = 0; j < NR; ++j) p[j] = mfma_bf16(w_0, h[j][kb], p[j]);
          w_0 = w_1;
          w_1 = w_2;
          __builtin_amdgcn_sched_barrier(0);
        }
        if constexpr (!PIPE && NR == 2) __builtin_amdgcn_s_setprio(0);
        u32x4 f[NR][2];
#pragma unroll
        for (int j = 0; j < NR; ++j) relu_to_frags(p[j], f[j][0], f[j][1]);
#pragma unroll
        for (int To = 0; To < AT; ++To) {
          const u32x4 wa = w3[(To * KH + 2 * cc) * 64 + ln];
          const u32x4 wb = w3[(To * KH + 2 * cc + 1) * 64 + ln];
#pragma unroll
          for (int j = 0; j < NR; ++j) {
            o[j][To] = mfma_bf16(wa, f[j][0], o[j][To]);
            o[j][To] = mfma_bf16(wb, f[j][1], o[j][To]);
          }
        }
      }
    }
    const int32_t un = u + NW;
#pragma unroll
    for (int j = 0; j < NR; ++j) epilogue<AT, RL>(a, c[j], o[j], nullptr, gg);
    if (un >= ur.end) break;
    u = un;
    if constexpr (PIPE) setup(u, first_loads(u), c, x, gg);
  }
}

// ---------------------------------------------------------------------------
// Streaming variant for wide three-layer policies whose weights do not fit in
// LDS (c3: 193 -> 512 -> 512 -> 64, 784 KB in bf16).
//
// A block of NW waves routes NW x 32 rows per step; each wave keeps its
// rows' whole first hidden layer in registers as bf16 B fragments. The
// weights pass through a double-buffered LDS ring in stages: two layer-1
// output tiles, or one layer-2 output tile together with the layer-3
// fragments that consume it (layer-2 outputs are never stored). The next
// stage is brought in by the LDS DMA path (global_load_lds, no registers)
// while the current one is multiplied; one barrier per stage.
// ---------------------------------------------------------------------------

// One 1 KB fragment (64 lanes x 16 B) from global memory into LDS; `dst` is
// wave-uniform, lane l's 16 bytes land at dst + 16 l.
__device__ __forceinline__ void dma_frag(u32x4* dst, const u32x4* src, int lane) {
  __builtin_amdgcn_global_load_lds((const void*)(src + lane),
                                   (__attribute__((address_space(3))) void*)dst, 16, 0, 0);
}

// 16 floats from LDS as four 16-byte reads (each keeps the LDS variable's
// alias information, which a single 64-byte access loses when it is split).
__device__ __forceinline__ f32x16 lds_f32x16(const u32x4* p) {
  const u32x4 v0 = p[0], v1 = p[1], v2 = p[2], v3 = p[3];
  f32x16 r;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    r[i] = __uint_as_float(v0[i]);
    r[4 + i] = __uint_as_float(v1[i]);
    r[8 + i] = __uint_as_float(v2[i]);
    r[12 + i] = __uint_as_float(v3[i]);
  }
  return r;
}

template <int H, int AT, int KB1, int ED, int NW, int RL>
__global__ __launch_bounds__(NW * 64, 1) void route_bf16_stream(RouteArgs a_in) {
  // chain pools: the tick's row count is on the device
  RouteArgs a = a_in;
  if (a_in.n_total_dev) a.n_total = min(*a_in.n_total_dev, a_in.n_total);   // the caller's buffers bound it
  constexpr int TH = H / 32, KH = H / 16;
  constexpr int S1 = TH / 2;                  // layer-1 stages (two output tiles each)
  constexpr int NST = S1 + TH;                // stages per block step
  constexpr int F1 = 2 * KB1;                 // fragments of a layer-1 stage
  constexpr int F2 = KH + 2 * AT;             // fragments of a layer-2 stage
  constexpr int FS = F1 > F2 ? F1 : F2;
  constexpr int NB0 = TH * 32, NB1 = TH * 32, NB2 = AT * 32;
  static_assert(NST % 2 == 0, "stage parity must repeat every block step");
  static_assert(KH % NW == 0 && 2 * AT <= NW, "layer-2 stage split over the waves");
  // Two separately declared buffers, each with its own copy of the biases
  // behind the weight fragments: a stage reads only the buffer the copy in
  // flight does not target, which the compiler can then tell apart (with one
  // array it waits for the next stage's copy before every read).
  constexpr int NBW = (NB0 + NB1 + NB2) / 4;   // biases in 16-byte words
  static_assert((NB0 + NB1 + NB2) % 4 == 0, "bias rows move in 16-byte words");
  __shared__ u32x4 ring0[FS * 64 + NBW];
  __shared__ u32x4 ring1[FS * 64 + NBW];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 5;
  const u32x4* W1 = (const u32x4*)a.W[0];
  const u32x4* W2 = (const u32x4*)a.W[1];
  const u32x4* W3 = (const u32x4*)a.W[2];
  // Fragments of stage st into ring buffer b: wave wv copies fragments
  // wv, wv + NW, ...; a wave with fewer fragments than the others copies the
  // stage's last one again (the same bytes to the same place), so the code
  // has no branches.
  auto issue = [&](int st, int b, int wv, int ln) {
    u32x4* dst = b ? ring1 : ring0;
    if (st < S1) {
#pragma unroll
      for (int i = 0; i < (F1 + NW - 1) / NW; ++i) {
        const int f = min(wv + NW * i, F1 - 1);
        dma_frag(dst + f * 64, W1 + (st * F1 + f) * 64, ln);
      }
    } else {
      const int j = st - S1;
#pragma unroll
      for (int i = 0; i < KH / NW; ++i) {
        const int f = wv + NW * i;
        dma_frag(dst + f * 64, W2 + (j * KH + f) * 64, ln);
      }
      const int f3 = min(wv, 2 * AT - 1);   // layer-3 fragment (To, 2 j + d) with f3 = 2 To + d
      dma_frag(dst + (KH + f3) * 64, W3 + ((f3 >> 1) * KH + 2 * j + (f3 & 1)) * 64, ln);
    }
  };
  for (int i = threadIdx.x; i < NB0 + NB1 + NB2; i += NW * 64) {
    const float v = i < NB0 ? a.bias[0][i] : (i < NB0 + NB1 ? a.bias[1][i - NB0] : a.bias[2][i - NB0 - NB1]);
    ((float*)(ring0 + FS * 64))[i] = v;
    ((float*)(ring1 + FS * 64))[i] = v;
  }
  issue(0, 0, __builtin_amdgcn_readfirstlane(wave), lane);
  // The block takes an equal contiguous share of the 32-row wave tiles (the
  // shares differ by at most one), NW per block step; in its last step the
  // waves without a tile still bring in their share of the weights and join
  // the barriers, but skip the arithmetic.
  const UnitRange ur = block_units((a.n_total + 31) / 32);
  const int n_steps = (ur.end - ur.first + NW - 1) / NW;
  for (int step = 0; step < n_steps; ++step) {
    // Per-iteration copies of the lane and wave indices: the fragment and
    // bias addresses derived from them are recomputed in each block step
    // instead of being hoisted out of the loop and kept live across it.
    asm volatile("" ::: "memory");
    int ln = lane, gg = g;
    int wv = __builtin_amdgcn_readfirstlane(wave);
    asm volatile("" : "+v"(ln), "+v"(gg));
    asm volatile("" : "+s"(wv));
    const int32_t unit = ur.first + step * NW + wv;
    const bool act = unit < ur.end;                             // wave-uniform
    const int32_t r0 = act ? unit * 32 : a.n_total - 1;        // idle waves: a clamped row, nothing stored
    const int32_t rl = r0 + 31 < a.n_total ? r0 + 31 : a.n_total - 1;
    const int32_t rows[1] = {act ? r0 + (ln & 31) : a.n_total};
    const int32_t rsel[1] = {rows[0] < a.n_total ? rows[0] : a.n_total - 1};
    int32_t envs[1];
    RowCtx c;
    u32x4 x[KB1];
    if (act) {
      find_envs<1>(a, r0, rl, rsel, envs);
      ValidRaw vr;
      c = row_setup_env_raw(a, rows[0], envs[0], vr);
      TailRaw<ED, KB1> raw;
      gather_issue<ED, KB1>(a, c, gg, x, raw);
      c.amask = mask_of(a, vr);
      gather_finish<ED, KB1>(a, c, gg, x, raw);
    }
    if (!act) {
      // the same stages, barriers and copies as a working wave (a barrier
      // counts waves, wherever they wait), without the arithmetic
      for (int s = 0; s < NST; ++s) {
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        int lns = ln;
        asm volatile("" : "+v"(lns));
        issue(s + 1 < NST ? s + 1 : 0, (s + 1) & 1, wv, lns);
      }
      continue;
    }
    u32x4 h[KH];
    f32x16 z[AT];
#pragma unroll
    for (int s = 0; s < NST; ++s) {
      // stage s is in buffer s & 1; every wave is done with buffer (s + 1) & 1
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      {
        // the DMA source addresses are formed here, not hoisted to the step's start
        int lns = ln;
        asm volatile("" : "+v"(lns));
        issue(s + 1 < NST ? s + 1 : 0, (s + 1) & 1, wv, lns);
      }
      const u32x4* wb = (s & 1) ? ring1 : ring0;
      const u32x4* lb4 = wb + FS * 64;   // biases, 4 floats per word
      if (s < S1) {
        // fragment q = t * KB1 + kb, two LDS reads ahead of its MFMA
        u32x4 w_0 = wb[0 * 64 + ln];
        u32x4 w_1 = wb[1 * 64 + ln];
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int T = 2 * s + t;
          f32x16 p = lds_f32x16(lb4 + (T * 2 + gg) * 4);
#pragma unroll
          for (int kb = 0; kb < KB1; ++kb) {
            const int q = t * KB1 + kb;
            const u32x4 w_2 = wb[(q + 2 < F1 ? q + 2 : F1 - 1) * 64 + ln];
            p = mfma_bf16(w_0, x[kb], p);
            w_0 = w_1;
            w_1 = w_2;
            __builtin_amdgcn_sched_barrier(0);
          }
          relu_to_frags(p, h[2 * T], h[2 * T + 1]);
        }
        if (s == S1 - 1) {
#pragma unroll
          for (int To = 0; To < AT; ++To) z[To] = lds_f32x16(lb4 + (NB0 + NB1) / 4 + (To * 2 + gg) * 4);
        }
      } else {
        const int j = s - S1;
        f32x16 p = lds_f32x16(lb4 + NB0 / 4 + (j * 2 + gg) * 4);
        u32x4 w_0 = wb[0 * 64 + ln];
        u32x4 w_1 = wb[1 * 64 + ln];
#pragma unroll
        for (int kb = 0; kb < KH; ++kb) {
          const u32x4 w_2 = wb[(kb + 2 < F2 ? kb + 2 : F2 - 1) * 64 + ln];
          p = mfma_bf16(w_0, h[kb], p);
          w_0 = w_1;
          w_1 = w_2;
          __builtin_amdgcn_sched_barrier(0);
        }
        u32x4 f0, f1;
        relu_to_frags(p, f0, f1);
        // w_0, w_1 now hold fragments KH and KH + 1 (layer 3, To = 0)
#pragma unroll
        for (int To = 0; To < AT; ++To) {
          const u32x4 wa = To == 0 ? w_0 : wb[(KH + 2 * To) * 64 + ln];
          const u32x4 wc = To == 0 ? w_1 : wb[(KH + 2 * To + 1) * 64 + ln];
          z[To] = mfma_bf16(wa, f0, z[To]);
          z[To] = mfma_bf16(wc, f1, z[To]);
        }
      }
    }
    epilogue<AT, RL>(a, c, z, nullptr, gg);
  }
  __builtin_amdgcn_s_waitcnt(0);   // the prefetched first stage of a step that does not exist
}

// ---------------------------------------------------------------------------
// The paper's dual-pathway executor (Sec. 4.2), persistent, on MFMA.
//
// Per request: a semantic pathway LN(ReLU(W_sem [e_q | e_r])) (128), a
// resource pathway LN(ReLU(W_res [h_bud | h_sys])) (64) over a budget head and
// a system head (16 each), a merge layer ReLU(W_merge [h_sem | h_res]) (128)
// and the action/value rows. The role half of the semantic layer takes only
// n_roles distinct inputs, so its products (plus b_sem) are computed once per
// pool (role_projection_kernel) and enter as the accumulator's initial value;
// the per-request semantic work is the 128 x E_d query half.
//
// A wave owns NR x 32 rows. The query-half, merge and action weights live in
// LDS (152 KB at E_d = 384); the small resource-layer fragments, the system
// head and the role projections are read through the caches. The query half
// of W_sem is packed so that each lane reads its row's embedding in 64-byte
// runs: within a 64-element group, lane half g takes elements 32 g .. 32 g + 31
// as four K steps of 8, so the two lanes of a row consume one 128-byte line
// per group. Groups are prefetched one ahead of the MFMAs that use them.
// ---------------------------------------------------------------------------

// fp32 -> bf16 (round to nearest even) -> fp32.
__device__ __forceinline__ float bf16_round(float x) { return __uint_as_float(pack2(x, 0.f) << 16); }

// ReLU, then LayerNorm over the 32 NT features a lane pair (n, n + 32) holds
// in NT accumulator tiles: (u - mean) / sqrt(var + 1e-5) * gain + bias with
// the biased variance, rounded to bf16 B fragments for the next layer
// (fragment 2T + h holds registers 8h .. 8h + 7 of tile T).
template <int NT>
__device__ __forceinline__ void relu_ln_frags(f32x16 (&acc)[NT], const float* gain, const float* bias,
                                              int g, u32x4 (&f)[2 * NT]) {
  constexpr float inv_n = 1.f / (32 * NT);
  float s = 0.f;
#pragma unroll
  for (int T = 0; T < NT; ++T) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      acc[T][v] = relu(acc[T][v]);
      s += acc[T][v];
    }
  }
  s += __shfl_xor(s, 32, 64);
  const float mean = s * inv_n;
  float q = 0.f;
#pragma unroll
  for (int T = 0; T < NT; ++T) {
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const float d = acc[T][v] - mean;
      q = fmaf(d, d, q);
    }
  }
  q += __shfl_xor(q, 32, 64);
  const float rstd = rsqrtf(fmaf(q, inv_n, 1e-5f));
#pragma unroll
  for (int T = 0; T < NT; ++T) {
    // one tile's gains and biases at a time: loads hoisted above this point
    // would keep all of them live at once
    asm volatile("" ::: "memory");
    float y[16];
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int i = (T * 2 + g) * 16 + v;
      y[v] = fmaf((acc[T][v] - mean) * rstd, gain[i], bias[i]);
    }
    f[2 * T].x = pack2(y[0], y[1]);     f[2 * T].y = pack2(y[2], y[3]);
    f[2 * T].z = pack2(y[4], y[5]);     f[2 * T].w = pack2(y[6], y[7]);
    f[2 * T + 1].x = pack2(y[8], y[9]);   f[2 * T + 1].y = pack2(y[10], y[11]);
    f[2 * T + 1].z = pack2(y[12], y[13]); f[2 * T + 1].w = pack2(y[14], y[15]);
    // the tile's fragments are complete before the next tile's loads issue
    asm volatile("" : "+v"(f[2 * T]), "+v"(f[2 * T + 1]));
  }
}

// The 4 K-step fragments of 64-element group G of a row's query embedding.
template <int ED>
__device__ __forceinline__ void load_group(const RouteArgs& a, const RowCtx& c, int G, int g, u32x4 (&x)[4]) {
  const u32x4* src = (const u32x4*)((const uint16_t*)a.emb + (size_t)c.q * ED + 64 * G + 32 * g);
#pragma unroll
  for (int i = 0; i < 4; ++i) x[i] = src[i];
}

// 64-element embedding groups in flight ahead of the MFMAs
constexpr int kDualPrefetch = 1;

template <int ED, int NW, int NR, int RL>
__global__ __launch_bounds__(NW * 64, 1) void route_dual_bf16(RouteArgs a_in) {
  // chain pools: the tick's row count is on the device
  RouteArgs a = a_in;
  if (a_in.n_total_dev) a.n_total = min(*a_in.n_total_dev, a_in.n_total);   // the caller's buffers bound it
  static_assert(ED % 64 == 0, "embedding width must be a multiple of 64");
  constexpr int KBQ = ED / 16;          // K steps of the query half
  constexpr int NG = ED / 64;           // 64-element groups
  constexpr int N_SEM = 4 * KBQ * 64;   // 16-byte fragments
  constexpr int N_MRG = 4 * 12 * 64;
  constexpr int N_ACT = 8 * 64;
  constexpr int WROWS = 32 * NR;
  __shared__ u32x4 lds[N_SEM + N_MRG + N_ACT];
  __shared__ float lp[DP_LDS];
  copy_to_lds<N_SEM, NW * 64>(lds, (const u32x4*)a.W[0]);
  copy_to_lds<N_MRG, NW * 64>(lds + N_SEM, (const u32x4*)a.W[1]);
  copy_to_lds<N_ACT, NW * 64>(lds + N_SEM + N_MRG, (const u32x4*)a.W[2]);
  for (int i = threadIdx.x; i < DP_LDS; i += NW * 64) lp[i] = a.dual_p[i];
  __syncthreads();
  const u32x4* wsem = lds;
  const u32x4* wmrg = lds + N_SEM;
  const u32x4* wact = wmrg + N_MRG;
  const u32x4* wres = (const u32x4*)a.W_res;
  const float* proj = a.dual_p + DP_ROLE;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n = lane & 31, g = lane >> 5;
  const int n3 = 3 * a.M;
  const int sstride = snap_stride(a.M);
  const UnitRange ur = block_units((a.n_total + WROWS - 1) / WROWS);

  for (int32_t u = ur.first + wave; u < ur.end; u += NW) {
    asm volatile("" ::: "memory");
    int ln = lane, gg = g;
    asm volatile("" : "+v"(ln), "+v"(gg));
    const int32_t r0 = u * WROWS;
    const int32_t rlast = (r0 + WROWS - 1 < a.n_total ? r0 + WROWS - 1 : a.n_total - 1);
    int32_t rows[NR], envs[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) rows[j] = r0 + 32 * j + n;
    find_envs<NR>(a, r0, rlast, rows, envs);
    RowCtx c[NR];
    int32_t role[NR];
    ValidRaw vr[NR];
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      c[j] = row_setup_env_raw(a, rows[j], envs[j], vr[j]);
      const int32_t ro = a.role[c[j].live ? rows[j] : a.n_total - 1];
      const bool bad_r = ro < 0 || ro >= a.n_roles;
      if (bad_r) c[j].bad |= IM_ERR_ROLE;
      role[j] = bad_r ? 0 : ro;
    }

    // ---- semantic pathway: role projection + W_sem (query half) e_q ----
    // ring of PF + 1 groups: group G + PF is loaded while group G is multiplied
    constexpr int PF = kDualPrefetch < NG ? kDualPrefetch : NG - 1;
    u32x4 x[PF + 1][NR][4];
#pragma unroll
    for (int G = 0; G < PF; ++G) {
#pragma unroll
      for (int j = 0; j < NR; ++j) load_group<ED>(a, c[j], G, gg, x[G][j]);
    }
#pragma unroll
    for (int j = 0; j < NR; ++j) c[j].amask = mask_of(a, vr[j]);
    // ---- resource pathway, computed while the first embedding groups load ----
    u32x4 hr[NR][4];
#pragma unroll
    for (int j = 0; j < NR; ++j) {
      // budget head: features 8 gg .. 8 gg + 7 of h_bud (K step 0 of W_res)
      const float bfe = bf16_round((float)c[j].budget * a.inv_bud);
      float hb[8], hy[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        hb[k] = relu(fmaf(lp[DP_W_BUD + 8 * gg + k], bfe, lp[DP_B_BUD + 8 * gg + k]));
        hy[k] = lp[DP_B_SYS + 8 * gg + k];
      }
      // system head: features 8 gg .. 8 gg + 7 of h_sys (K step 1) over the
      // env's queue-depth, KV-proxy and latency features, read 8 at a time
      // (weights of the features past 3M are zero)
      const float* srow = a.snap + (size_t)c[j].e * sstride;
      for (int k0 = 0; k0 < n3; k0 += 8) {
        const float4 d0 = *(const float4*)(srow + k0);
        const float4 d1 = *(const float4*)(srow + k0 + 4);
        const float dv[8] = {d0.x, d0.y, d0.z, d0.w, d1.x, d1.y, d1.z, d1.w};
#pragma unroll
        for (int kk = 0; kk < 8; ++kk) {
          const float d = bf16_round(dv[kk]);
          const float* w = lp + DP_W_SYS + (k0 + kk) * 16 + 8 * gg;
#pragma unroll
          for (int q = 0; q < 8; ++q) hy[q] = fmaf(w[q], d, hy[q]);
        }
      }
      u32x4 f0, f1;
      f0.x = relu_pack2(hb[0], hb[1]); f0.y = relu_pack2(hb[2], hb[3]);
      f0.z = relu_pack2(hb[4], hb[5]); f0.w = relu_pack2(hb[6], hb[7]);
      f1.x = relu_pack2(hy[0], hy[1]); f1.y = relu_pack2(hy[2], hy[3]);
      f1.z = relu_pack2(hy[4], hy[5]); f1.w = relu_pack2(hy[6], hy[7]);
      f32x16 rr[2];
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        rr[T] = *(const f32x16*)(lp + DP_B_RES + (T * 2 + gg) * 16);
        rr[T] = mfma_bf16(wres[(T * 2 + 0) * 64 + ln], f0, rr[T]);
        rr[T] = mfma_bf16(wres[(T * 2 + 1) * 64 + ln], f1, rr[T]);
      }
      relu_ln_frags<2>(rr, lp + DP_LN_RES_G, lp + DP_LN_RES_B, gg, hr[j]);
    }
    __builtin_amdgcn_sched_barrier(0);

    f32x16 s[NR][4];
#pragma unroll
    for (int j = 0; j < NR; ++j) {
#pragma unroll
      for (int T = 0; T < 4; ++T) s[j][T] = *(const f32x16*)(proj + ((role[j] * 4 + T) * 2 + gg) * 16);
    }
#pragma unroll
    for (int G = 0; G < NG; ++G) {
      if (G + PF < NG) {
#pragma unroll
        for (int j = 0; j < NR; ++j) load_group<ED>(a, c[j], G + PF, gg, x[(G + PF) % (PF + 1)][j]);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kb = 4 * G + i;
#pragma unroll
        for (int T = 0; T < 4; ++T) {
          const u32x4 w = wsem[(T * KBQ + kb) * 64 + ln];
#pragma unroll
          for (int j = 0; j < NR; ++j) s[j][T] = mfma_bf16(w, x[G % (PF + 1)][j][i], s[j][T]);
        }
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    u32x4 hs[NR][8];
#pragma unroll
    for (int j = 0; j < NR; ++j) relu_ln_frags<4>(s[j], lp + DP_LN_SEM_G, lp + DP_LN_SEM_B, gg, hs[j]);
    __builtin_amdgcn_sched_barrier(0);

    // ---- decision: merge layer, then the action/value rows ----
    u32x4 hh[NR][8];
#pragma unroll
    for (int T = 0; T < 4; ++T) {
      f32x16 m[NR];
      m[0] = *(const f32x16*)(lp + DP_B_MERGE + (T * 2 + gg) * 16);
#pragma unroll
      for (int j = 1; j < NR; ++j) m[j] = m[0];
#pragma unroll
      for (int kb = 0; kb < 12; ++kb) {
        const u32x4 w = wmrg[(T * 12 + kb) * 64 + ln];
#pragma unroll
        for (int j = 0; j < NR; ++j) m[j] = mfma_bf16(w, kb < 8 ? hs[j][kb] : hr[j][kb - 8], m[j]);
      }
#pragma unroll
      for (int j = 0; j < NR; ++j) relu_to_frags(m[j], hh[j][2 * T], hh[j][2 * T + 1]);
      __builtin_amdgcn_sched_barrier(0);
    }
    f32x16 o[NR][1];
    o[0][0] = *(const f32x16*)(lp + DP_B_ACT + gg * 16);
#pragma unroll
    for (int j = 1; j < NR; ++j) o[j][0] = o[0][0];
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) {
      const u32x4 w = wact[kb * 64 + ln];
#pragma unroll
      for (int j = 0; j < NR; ++j) o[j][0] = mfma_bf16(w, hh[j][kb], o[j][0]);
    }
#pragma unroll
    for (int j = 0; j < NR; ++j) epilogue<1, RL>(a, c[j], o[j], nullptr, gg);
  }
}

// Role projections, one thread per (role, output feature): fp32 sum of the
// bf16 products, stored in accumulator-register order.
__global__ void role_projection_kernel(const uint16_t* w_role, const uint16_t* roles, const float* b_sem,
                                       int n_roles, int ed, float* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= n_roles * kDualSem) return;
  const int r = i / kDualSem, o = i % kDualSem;
  float acc = b_sem[o];
  for (int k = 0; k < ed; ++k)
    acc = fmaf(bf16_to_f32(w_role[(size_t)o * ed + k]), bf16_to_f32(roles[(size_t)r * ed + k]), acc);
  // feature o = 32 T + 8 (v / 4) + 4 g + v % 4
  const int T = o >> 5, w = o & 31, v = ((w >> 3) << 2) | (w & 3), g = (w >> 2) & 1;
  out[(((size_t)r * 4 + T) * 2 + g) * 16 + v] = acc;
}

typedef void (*RouteKernel)(RouteArgs);

template <int H, int NL>
RouteKernel pick_bf16(int at) {
  return at == 1 ? route_bf16<H, NL, 1> : (at == 2 ? route_bf16<H, NL, 2> : route_bf16<H, NL, 3>);
}
template <int H, int NL>
RouteKernel pick_f32(int at) {
  // at: output tiles of 16 (fp32 pools); feature-split kernel when the hidden
  // tiles split four ways
  if constexpr ((H / 16) % 4 == 0)
    return at == 1 ? route_f32s<H, NL, 1>
                   : (at == 2 ? route_f32s<H, NL, 2> : (at == 3 ? route_f32s<H, NL, 3> : route_f32s<H, NL, 4>));
  return at == 1 ? route_f32<H, NL, 1>
                 : (at == 2 ? route_f32<H, NL, 2> : (at == 3 ? route_f32<H, NL, 3> : route_f32<H, NL, 4>));
}

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

// Persistent LDS-resident kernels and their launch shape (waves per block,
// 32-row MFMA tiles per wave). The greedy route and the RL outputs are
// separate instantiations, so each keeps only the registers its own epilogue
// needs.
struct LdsLaunch {
  RouteKernel k;
  int waves;   // per block
  int rows;    // 32-row MFMA tiles per wave
};

// 86 -> 256 -> 256 -> A, layer-1 weights through the caches: the greedy
// route runs 8 waves (two per SIMD) of 64 rows, so every weight fragment read
// from LDS or the caches feeds two MFMAs, with the next output tile's layer-1
// fragments loaded while the current one is multiplied (up to 256 VGPRs per
// wave); the RL outputs, whose epilogue needs more registers, and light
// ticks, whose few tiles would leave most waves idle, run 16 waves of 32
// rows; very light ticks 8 waves of 32 rows, software-pipelined.
// 104 -> 256 -> A, every layer in LDS, software-pipelined, the output layer
// consuming each hidden tile as soon as it is produced: the greedy route runs
// 12 waves (three per SIMD, 168 VGPRs) of 64 rows, so each weight fragment
// read from LDS feeds two MFMAs; the RL outputs run 16 waves of 32 rows (102
// VGPRs). Returns a null kernel when no LDS-resident variant applies.
LdsLaunch pick_lds(int dtype, int hidden, int n_layers, int out_tiles, int k1, int ed, bool rl, int light) {
  if (dtype != IM_BF16) return {nullptr, 0, 0};
  if (hidden == 256 && n_layers == 3 && out_tiles == 1 && k1 == 6 && ed == 64) {
    if (rl) return {route_bf16_lds<256, 3, 1, 6, false, 16, 64, 1, 1, 0, false>, 16, 1};
    if (light == 2) return {route_bf16_lds<256, 3, 1, 6, false, 8, 64, 1, 0, 6, true>, 8, 1};
    if (light == 1) return {route_bf16_lds<256, 3, 1, 6, false, 16, 64, 1, 0, 0, false>, 16, 1};
    return {route_bf16_lds<256, 3, 1, 6, false, 8, 64, 2, 0, 6, false>, 8, 2};
  }
  if (hidden == 256 && n_layers == 2 && out_tiles == 1 && k1 == 7 && ed == 64)
    return {rl ? route_bf16_lds<256, 2, 1, 7, true, 16, 64, 1, 1, 0, true>
               : route_bf16_lds<256, 2, 1, 7, true, 12, 64, 2, 0, 0, true>, rl ? 16 : 12, rl ? 1 : 2};
  return {nullptr, 0, 0};
}

// Streaming kernels: kStreamWaves waves per block, 32 rows per wave. The
// greedy route and the RL outputs are separate instantiations, so each keeps
// only the registers its own epilogue needs.
constexpr int kStreamWaves = 8;

RouteKernel pick_stream(int dtype, int hidden, int n_layers, int out_tiles, int k1, int ed, bool rl) {
  if (dtype != IM_BF16) return nullptr;
  if (hidden == 512 && n_layers == 3 && out_tiles == 2 && k1 == 13 && ed == 128)
    return rl ? route_bf16_stream<512, 2, 13, 128, kStreamWaves, 1>
              : route_bf16_stream<512, 2, 13, 128, kStreamWaves, 0>;
  if (hidden == 512 && n_layers == 3 && out_tiles == 3 && k1 == 13 && ed == 128)
    return rl ? route_bf16_stream<512, 3, 13, 128, kStreamWaves, 1>
              : route_bf16_stream<512, 3, 13, 128, kStreamWaves, 0>;
  return nullptr;
}

// Dual-pathway kernels: kDualWaves waves per block, kDualRows row tiles per wave.
constexpr int kDualWaves = 16;
constexpr int kDualRows = 1;

RouteKernel pick_dual(int ed, bool rl) {
  switch (ed) {
    case 64: return rl ? route_dual_bf16<64, kDualWaves, kDualRows, 1> : route_dual_bf16<64, kDualWaves, kDualRows, 0>;
    case 128: return rl ? route_dual_bf16<128, kDualWaves, kDualRows, 1> : route_dual_bf16<128, kDualWaves, kDualRows, 0>;
    case 256: return rl ? route_dual_bf16<256, kDualWaves, kDualRows, 1> : route_dual_bf16<256, kDualWaves, kDualRows, 0>;
    case 384: return rl ? route_dual_bf16<384, kDualWaves, kDualRows, 1> : route_dual_bf16<384, kDualWaves, kDualRows, 0>;
  }
  return nullptr;
}

hipError_t launch_dual(const RouteArgs& a, hipStream_t s) {
  RouteKernel k = pick_dual(a.embed_dim, a.rl != 0);
  if (!k) return hipErrorInvalidValue;
  const int rows = 32 * kDualRows;
  const int units = (a.n_total + rows - 1) / rows;   // wave tiles, spread over up to one block per CU
  const unsigned blocks =
      (unsigned)(a.persistent_blocks > 0 && units > a.persistent_blocks ? a.persistent_blocks : units);
  hipLaunchKernelGGL(k, dim3(blocks), dim3(kDualWaves * 64), 0, s, a);
  return hipGetLastError();
}

}  // namespace

bool dual_supported(int embed_dim, int out_rows) {
  return out_rows >= 1 && out_rows <= 32 && pick_dual(embed_dim, false) != nullptr;
}

hipError_t launch_role_projection(const uint16_t* w_role, const uint16_t* roles, const float* b_sem,
                                  int n_roles, int embed_dim, float* out, hipStream_t s) {
  const int n = n_roles * kDualSem;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(role_projection_kernel, dim3((n + 255) / 256), dim3(256), 0, s, w_role, roles, b_sem,
                     n_roles, embed_dim, out);
  return hipGetLastError();
}

// out_tiles: output tiles of the last layer, 32 rows (bf16) or 16 rows (fp32).
bool route_supported(int dtype, int hidden, int n_layers, int out_tiles) {
  if (out_tiles < 1 || out_tiles > (dtype == IM_F32 ? 4 : 3)) return false;
  RouteKernel k = n_layers == 2 ? pick<2>(dtype, hidden, out_tiles)
                 : n_layers == 3 ? pick<3>(dtype, hidden, out_tiles) : nullptr;
  return k != nullptr;
}

hipError_t launch_route(const RouteArgs& a, int dtype, int hidden, int n_layers, int out_tiles,
                        hipStream_t s) {
  if (a.n_total <= 0) return hipSuccess;
  if (a.net == IM_NET_DUAL) return launch_dual(a, s);
  if (a.persistent_blocks > 0) {
    // a light tick (at most three 64-row tiles per four waves of 8-wave
    // blocks) runs the 16-wave, 32-row shape: twice the waves share its rows;
    // a very light one (at most one 32-row tile per two waves) runs 8 waves
    // of 32 rows whose first tile's loads overlap the block's weight copy
    const int64_t rows = a.n_total, cap = (int64_t)64 * 8 * a.persistent_blocks;
    const int light = rows * 4 <= cap ? 2 : (rows * 4 <= 3 * cap ? 1 : 0);
    const LdsLaunch kl = pick_lds(dtype, hidden, n_layers, out_tiles, a.k1, a.embed_dim, a.rl != 0, light);
    if (kl.k) {
      // one block per CU as long as there are wave tiles for them: a light
      // tick spreads its few tiles over every CU instead of filling a few
      const int rows = 32 * kl.rows;
      const int units = (a.n_total + rows - 1) / rows;
      const unsigned blocks = (unsigned)(units < a.persistent_blocks ? units : a.persistent_blocks);
      hipLaunchKernelGGL(kl.k, dim3(blocks), dim3(kl.waves * 64), 0, s, a);
      return hipGetLastError();
    }
  }
  if (a.persistent_blocks > 0) {
    RouteKernel ks = pick_stream(dtype, hidden, n_layers, out_tiles, a.k1, a.embed_dim, a.rl != 0);
    if (ks) {
      const int rows = kStreamWaves * 32;
      const int n_tiles = (a.n_total + rows - 1) / rows;
      const unsigned blocks = (unsigned)(n_tiles < a.persistent_blocks ? n_tiles : a.persistent_blocks);
      hipLaunchKernelGGL(ks, dim3(blocks), dim3(kStreamWaves * 64), 0, s, a);
      return hipGetLastError();
    }
  }
  RouteKernel k = nullptr;
  if (route_supported(dtype, hidden, n_layers, out_tiles)) {
    if (n_layers == 2) k = pick<2>(dtype, hidden, out_tiles);
    else if (n_layers == 3) k = pick<3>(dtype, hidden, out_tiles);
  }
  if (!k) return hipErrorInvalidValue;
  if (a.n_total <= 0) return hipSuccess;
  // blocks of 4 waves: 32 rows per wave (bf16), 16 rows per wave (fp32,
  // hidden width 32) or 16 rows per block (fp32, feature-split)
  const int rows = dtype == IM_F32 ? (hidden % 64 == 0 ? 16 : 64) : 128;
  const unsigned blocks = (unsigned)((a.n_total + rows - 1) / rows);
  hipLaunchKernelGGL(k, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace im
