// Internal device data layout and kernel argument blocks of libinframind.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "inframind.h"

namespace im {

// Per-(env, model) state, 64 bytes. The queue of a model is split into a
// sorted "front" (the smallest keys, at most kFront entries, occupying
// front[fh .. fh+fn)) and an unsorted "pool" of the rest (pool[0 .. P)).
// Every front key is smaller than every pool key; qlen = fn + P.
struct alignas(64) ModelRec {
  int32_t qlen, busy, ewma, backlog;   // snapshot fields read by the route step
  int32_t cap, enabled, fh, fn;
  int32_t P;
  int32_t next_id, t;                  // the env's next request id and ticks completed
                                       // (kept in the env's first record only)
  int32_t busy_mask;                   // bit s: slot s busy
  int32_t next_done;                   // earliest completion tick of a busy slot
  int32_t rpm_limit;                   // blackbox rate limit per kRpmWindow ticks (0: none)
  int32_t rpm_count;                   // dispatches in the last kRpmWindow ticks
  float inv_rpm;                       // 1 / rpm_limit rounded once to fp32
};
static_assert(sizeof(ModelRec) == 64, "ModelRec layout");

constexpr int kFront = 64;       // front capacity (one entry per lane)
constexpr int kRpmWindow = 60;   // blackbox dispatch window (ticks; App. C: 60 s)
constexpr int kRpmRing = 64;     // bytes per (env, model) of the per-tick dispatch ring

// Per-env snapshot row read by the route step, written by the schedule step
// (and by snapshot_kernel after host-side state changes): the 4M load-stat
// features in stat-major order as fp32 (each one product of an integer and a
// reciprocal rounded once to fp32), then one validity byte per model (enabled,
// c_m > 0 and queue below capacity), padded so 8 consecutive floats can always
// be read from any feature index < 4M.
__host__ __device__ inline int snap_stride(int M) {
  const int n = 4 * M + (M + 3) / 4 + 8;
  return (n + 7) & ~7;
}
__host__ __device__ inline int snap_valid_offset(int M) { return 4 * M; }   // in floats

// Counter slots per (env, model), int64. C_COST_Q16 sums floor(2^16 latency /
// budget) over completions (the cost of Eq. 2, for the dual update of Eq. 7).
enum { C_REJ_OVERFLOW = 0, C_ENQUEUED, C_STARTED, C_COMPLETED, C_SLO_MET, C_LAT_SUM,
       C_WAIT_SUM, C_COST_Q16, C_NUM = 8 };

// Multi-step chains (Sec. 4.3): a call carries its query in two words that
// travel with its queue entry, its slot and its pending record:
//   A = q_idx | k << 24 | n_steps << 28   (call k of n_steps; q_idx < 2^24)
//   B = base_svc | beta << 12 | role0 << 27   (base_svc < 2^12, query budget
//       beta < 2^15, role of the first call < 32)
// A pending call (spawned by the completion of call k - 1, routed at the next
// tick) is {A, B, deadline, 0}. Env counters: arrived, rej_nomodel, completed
// queries, queries completed by their deadline.
constexpr int kMaxSteps = 15;
constexpr int kEnvCnt = 4;
enum { E_ARRIVED = 0, E_REJ_NOMODEL, E_Q_DONE, E_Q_MET };
__host__ __device__ inline int32_t chain_a(int32_t q_idx, int k, int n_steps) {
  return (int32_t)((uint32_t)q_idx | ((uint32_t)k << 24) | ((uint32_t)n_steps << 28));
}
__host__ __device__ inline int32_t chain_b(int base, int beta, int role0) {
  return (int32_t)(((uint32_t)base & 0xfffu) | (((uint32_t)beta & 0x7fffu) << 12) |
                   (((uint32_t)role0 & 31u) << 27));
}
__host__ __device__ inline int32_t chain_q(int32_t A) { return A & 0xffffff; }
__host__ __device__ inline int chain_k(int32_t A) { return (A >> 24) & 15; }
__host__ __device__ inline int chain_n(int32_t A) { return (int)((uint32_t)A >> 28); }
__host__ __device__ inline int chain_base(int32_t B) { return B & 0xfff; }
__host__ __device__ inline int chain_beta(int32_t B) { return (B >> 12) & 0x7fff; }
__host__ __device__ inline int chain_role0(int32_t B) { return (int)((uint32_t)B >> 27); }
// remaining budget of a call routed at tick t, in the int16 range of budgets
__host__ __device__ inline int32_t remaining_budget(int32_t deadline, int32_t t) {
  const int64_t b = (int64_t)deadline - t;
  return (int32_t)(b < -32768 ? -32768 : (b > 32767 ? 32767 : b));
}

// Queue entry in device memory: {key, id, t_arr, svc | budget << 16} (budget
// signed: a later call of a chain may be routed past its deadline).
// Slot in device memory: {id (-1 free), t_arr, tick at which it completes, budget};
// the state export reports the service ticks left instead of the completion tick.

// Dual-pathway executor (Sec. 4.2): fixed widths of the paper.
constexpr int kDualSem = 128, kDualBud = 16, kDualSys = 16, kDualRes = 64, kDualMerge = 128;
constexpr int kDualMaxModels = 16;   // the system head's weights are staged in LDS
// Its fp32 parameter block (offsets in floats). Vectors in accumulator-register
// order [tile][g][16] (feature 32 tile + 8 (v / 4) + 4 g + v % 4 at index
// (2 tile + g) 16 + v). The first DP_LDS floats are staged in LDS.
enum {
  DP_LN_SEM_G = 0,      // [128] semantic LayerNorm gain
  DP_LN_SEM_B = 128,    // [128] semantic LayerNorm bias
  DP_B_RES = 256,       // [64] resource layer bias
  DP_LN_RES_G = 320,    // [64] resource LayerNorm gain
  DP_LN_RES_B = 384,    // [64] resource LayerNorm bias
  DP_B_MERGE = 448,     // [128] merge bias
  DP_B_ACT = 576,       // [32] action/value bias (+ per-model logit bias on action rows)
  DP_W_BUD = 608,       // [16] budget head (natural order)
  DP_B_BUD = 624,       // [16]
  DP_B_SYS = 640,       // [16] system head bias (natural order)
  DP_W_SYS = 656,       // [3 kDualMaxModels][16]: W_sys column of snapshot feature k (zero
                        // for k >= 3M), rows 0..15
  DP_LDS = DP_W_SYS + 3 * kDualMaxModels * 16,
  DP_ROLE = DP_LDS      // [n_roles][4][2][16]: b_sem + W_sem[:, E_d:] e_r per role, in
                        // accumulator order
};

struct RouteArgs {
  const int32_t* offsets;
  const int32_t* q_idx;
  const int16_t* budget;
  int32_t n_total;
  float envs_per_row;                 // E / n_total: first guess of a row's env
  int32_t E, M, K, A;
  int32_t embed_dim, feat_dim, k1;    // k1: layer-1 K steps (bf16: 16-wide, f32: 2-wide)
  int32_t qcap;
  int64_t Q;
  const void* emb;
  const void* W[3];                   // packed weights per layer
  const float* bias[3];               // packed biases per layer (D-register order)
  const ModelRec* ms;
  const float* snap;                  // [E * snap_stride(M)]
  float inv_bud;
  int32_t* actions;
  float* logits;
  int32_t* err;
  int32_t persistent_blocks;          // grid of the persistent kernels (0: never use them)
  // RL-rollout outputs (im_route_sample)
  int32_t rl;                         // 1: log-prob, entropy, value; sampled or greedy action
  int32_t greedy;                     // with rl: 1 = masked argmax, 0 = Gumbel-max sample
  uint32_t seed_lo, seed_hi;          // Philox key
  float* logp;
  float* entropy;
  float* value;                       // row A of the last layer (value head), or NULL
  const int32_t* n_total_dev;         // chain pools: the tick's row count (device); n_total
                                      // then bounds it
  // dual-pathway executor (net == IM_NET_DUAL): W[0] semantic (query half),
  // W[1] merge, W[2] action/value fragments; W_res resource-layer fragments
  int32_t net;
  const int16_t* role;
  int32_t n_roles;
  const void* W_res;
  const float* dual_p;                // fp32 parameter block (DP_* offsets)
};

struct SchedArgs {
  const int32_t* offsets;
  const int32_t* q_idx;
  const int16_t* budget;
  const int16_t* base_svc;
  const int32_t* actions;   // per row: at offsets[e] + i, or (chains) roff[e] + i
  // multi-step chains: calls per arriving query, row offsets of the tick (the
  // env's pending calls, then its arrivals), pending calls and their counts
  // double-buffered by tick parity ([2][E * pend_cap], [2][E]), the ext words
  // (A, B) of queue entries and slots
  const int16_t* n_steps;
  int32_t max_steps, pend_cap;
  const int32_t* roff;
  int4* pend;
  int32_t* pcnt;
  int2* front_ext;
  int2* pool_ext;
  int2* slot_ext;
  const int32_t* csr_bad;   // chain pools: set when the rows build found the arrival CSR broken
  int32_t n_total;
  int32_t E, M, K, A, S, qcap, max_arrivals, key_mode;
  int64_t Q;
  ModelRec* ms;
  int64_t* cnt;       // [E*M*C_NUM]
  int64_t* env_cnt;   // [E*kEnvCnt] arrived, rej_nomodel, completed queries, on-time queries
  int64_t* hist;      // [E*A]
  int4* slots;        // [E*M*S]
  int4* front;        // [E*M*kFront]
  int4* pool;         // [E*M*qcap]
  uint8_t* rpm_ring;  // [E*M*kRpmRing]: dispatches at tick tau in byte tau % kRpmWindow
  const int16_t* role;  // per-row role (dual-pathway pools; NULL otherwise)
  int32_t n_roles;
  int32_t* err;
  float* snap;        // [E * snap_stride(M)]
  float inv_qcap, inv_lat;
  const float* inv_tab;  // [2*(IM_MAX_SLOTS+1)]: 1/max(c,1), then 1/(max(c,1)*budget_max)
};

// Host-side launchers (defined in the .hip files).
// Dual update (Eq. 7): acc [2] device accumulators (zero between calls), last
// [2] totals at the previous update, lambda device in/out.
// env_cnt (chain pools, else NULL): queries are counted from its completed-query
// column instead of the per-model completions.
hipError_t launch_dual_update(const int64_t* cnt, int64_t n_em, const int64_t* env_cnt, int64_t n_env,
                              unsigned long long* acc, int64_t* last, double eta, double lambda_max,
                              double* lambda, hipStream_t s);
bool route_supported(int dtype, int hidden, int n_layers, int out_tiles);
bool dual_supported(int embed_dim, int out_rows);
// Role projections of the dual-pathway executor: out[r][tile][g][16] =
// b_sem + W_sem[:, E_d:] e_r in fp32 for every role r (bf16 inputs).
//   w_role [128 x E_d] bf16 bits, roles [n_roles x E_d] bf16 bits, b_sem [128]
hipError_t launch_role_projection(const uint16_t* w_role, const uint16_t* roles, const float* b_sem,
                                  int n_roles, int embed_dim, float* out, hipStream_t s);
hipError_t launch_route(const RouteArgs& a, int dtype, int hidden, int n_layers, int out_tiles,
                        hipStream_t s);
// rpm: some model of the pool is (or was) rate-limited (blackbox windows tracked);
// waves_per_block: envs per block (1, 2 or 4)
hipError_t launch_schedule(const SchedArgs& a, bool rpm, bool chain, int waves_per_block, hipStream_t s);
// Rows of a chain pool's tick: row offsets (pending calls first, then the
// usable arrivals of each env), the row count and the route step's per-row
// inputs (q_idx, remaining budget, role of the call).
struct RowsArgs {
  const int32_t* offsets;   // arrival CSR [E+1]
  int32_t n_total, E, M, max_arrivals, pend_cap, n_roles;   // n_roles: 0 for MLP pools
  const int32_t* q_idx;
  const int16_t* budget;
  const int16_t* role;
  const ModelRec* ms;       // the tick: ms[0].t
  const int4* pend;         // [2][E * pend_cap]
  const int32_t* pcnt;      // [2][E]
  int32_t* roff;            // out [E+1]
  int32_t* n_rows;          // out [2]: the row count, then 1 when the arrival CSR is not
                            // one monotone partition of [0, n_total) (no arrival is then usable)
  int32_t* rq;              // out per row
  int16_t* rb;
  int16_t* rr;
};
hipError_t launch_rows(const RowsArgs& a, hipStream_t s);
// Recompute the snapshot rows of envs [e0, e0 + ne) from the model records.
hipError_t launch_snapshot(const SchedArgs& a, int e0, int ne, hipStream_t s);

}  // namespace im
