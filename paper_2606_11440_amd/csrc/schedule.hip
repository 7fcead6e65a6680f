// Schedule step of the tick: admission, queue insertion, service, accounting.
//
// One wave owns one env (all of its model queues); a block holds 4 such waves
// and the waves never synchronise with each other (no block barriers), so
// every wave runs its env independently.
//
// Per queue, in the order the tick defines:
//   admission  -- the env's routed requests for this model, in id order, are
//                 accepted while the queue has room (tail-drop beyond the
//                 capacity); stable partition by model = ballot + mbcnt.
//   keys       -- svc = base_svc * (depth + 1); key = t + budget - svc (slack,
//                 i.e. latest start time), t + budget (deadline, Sec. 4.3) or t
//                 (arrival order). The queue order is (key, id).
//   insertion  -- the queue is kept as a sorted front of at most 64 entries
//                 (one per lane, held in registers while the wave works on the
//                 queue) with the smallest keys, plus an unsorted pool of the
//                 rest. The env's arrivals are sorted 64 at a time by (model,
//                 key, id); a model's newcomers below the front's largest key
//                 are merged into the front with a bitonic merge network (its
//                 overflow spills to the pool), the others are appended to the
//                 pool. The front array is written once per tick, if changed.
//   service    -- free slots below c_m are filled in slot order from the front
//                 head; when the front runs empty it is refilled with the 64
//                 smallest pool entries (bitonic top-64 selection), and the
//                 pool is compacted. Busy slots then advance one tick; a
//                 request completes when its remaining time reaches 0 (latency
//                 EWMA with alpha = 1/8 in Q8, Sec. 5.4; bounded concurrency
//                 as in Table 5).
#include "im_internal.h"
#include "wave.h"

namespace im {
namespace {

constexpr int64_t kKeyMax = 0x7fffffffffffffffll;

__device__ __forceinline__ int64_t composite(int32_t key, int32_t id) {
  return (int64_t)(((uint64_t)(uint32_t)key << 32) | (uint32_t)id);
}
__device__ __forceinline__ int32_t comp_key(int64_t c) { return (int32_t)(c >> 32); }
__device__ __forceinline__ int32_t comp_id(int64_t c) { return (int32_t)(uint32_t)c; }

// Arrival tick of a queue entry from its key and packed (svc | budget << 16):
// the key is t_arr + budget - svc (slack), t_arr + budget (deadline) or t_arr
// (arrival order), so the arrival tick never has to travel with the entry
// through a sort network.
__device__ __forceinline__ int32_t t_arr_of(int32_t key, int32_t svcbud, int key_mode) {
  const uint32_t svc = (uint32_t)svcbud & 0xffffu, bud = (uint32_t)(svcbud >> 16);   // budget signed
  const uint32_t k = (uint32_t)key;
  return (int32_t)(key_mode == IM_KEY_DEADLINE ? k - bud : (key_mode == IM_KEY_FCFS ? k : k - bud + svc));
}

// A wave-uniform 32-bit load through the scalar data cache, for data no
// kernel of the tick writes while this one runs (the offsets, the rows
// build's results).
__device__ __forceinline__ int32_t load_uniform(const int32_t* p) {
  return *(const __attribute__((address_space(4))) int32_t*)p;
}

// Makes this wave's earlier global stores visible to its later loads.
__device__ __forceinline__ void wave_mem_sync() { __threadfence_block(); }

struct Queue {       // wave-uniform view of one (env, model) record
  int32_t qlen, busy, ewma, backlog, cap, enabled, fh, fn, P, busy_mask, next_done;
};

// Merge `lim` newcomers into the front held in registers (`fe`, lane i <
// q.fn), all of them below the front's largest key or the pool empty. `seg`
// is the model's sorted segment of a staged chunk in LDS (entries (key, id,
// svc | budget << 16, model)). Only the key and the packed service/budget word
// (and, with CHAIN, the two chain words: `fx`, `segx`, `pool_ext`) pass
// through the network; arrival ticks are recovered from them. The front followed
// by the reversed newcomers is a bitonic sequence of 128; its half-cleaner
// leaves the 64 smallest in `lo` (bitonic, sorted by one merge network) and
// the rest in `hi`, whose real entries spill to the pool.
template <bool CHAIN>
__device__ __forceinline__ void merge_front(Queue& q, int4& fe, int2& fx, const int4* seg,
                                            const int2* segx, int lim, int key_mode, int4* pool,
                                            int2* pool_ext) {
  constexpr int NP = CHAIN ? 3 : 1;
  const int lane = lane_id();
  const int r = 63 - lane;
  int64_t kb = kKeyMax;
  int32_t pb[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) pb[i] = 0;
  if (r < lim) {
    const int4 v = seg[r];
    kb = composite(v.x, v.y);
    pb[0] = v.z;
    if constexpr (CHAIN) {
      const int2 x = segx[r];
      pb[1] = x.x;
      pb[2] = x.y;
    }
  }
  const int64_t ka = lane < q.fn ? composite(fe.x, fe.y) : kKeyMax;
  int32_t pa[NP];
  pa[0] = fe.w;
  if constexpr (CHAIN) {
    pa[1] = fx.x;
    pa[2] = fx.y;
  }
  const bool sw = kb < ka;
  int64_t klo = sw ? kb : ka;
  const int64_t khi = sw ? ka : kb;
  int32_t plo[NP], phi[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    plo[i] = sw ? pb[i] : pa[i];
    phi[i] = sw ? pa[i] : pb[i];
  }
  bitonic_merge64<NP>(klo, plo);
  const int total = q.fn + lim;
  const int keep = total < kFront ? total : kFront;
  const bool spill = khi != kKeyMax;
  const uint64_t sm = ballot(spill);
  if (spill) {
    const int32_t kk = comp_key(khi);
    const int pos = q.P + prefix_count(sm);
    pool[pos] = make_int4(kk, comp_id(khi), t_arr_of(kk, phi[0], key_mode), phi[0]);
    if constexpr (CHAIN) pool_ext[pos] = make_int2(phi[1], phi[2]);
  }
  q.P += total - keep;
  q.fh = 0;
  q.fn = keep;
  const int32_t kl = comp_key(klo);
  fe = lane < keep ? make_int4(kl, comp_id(klo), t_arr_of(kl, plo[0], key_mode), plo[0])
                   : make_int4(0, 0, 0, 0);
  if constexpr (CHAIN) fx = lane < keep ? make_int2(plo[1], plo[2]) : make_int2(0, 0);
}

// Refill the (empty) front with the min(64, P) smallest pool entries; the new
// front is returned in `fe` (lane i: entry i), the front array is not written.
// `pk`/`pi` are this wave's LDS staging rows (64 keys, 64 pool indices), `kb`
// its LDS buffer for 4 chunks of pool keys.
// Pool chunks (of 64 entries) per round of the refill scan (chain pools,
// whose kernel holds more LDS, use fewer to keep 4 blocks per CU), and the
// s_waitcnt immediate (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// 6:4 and lgkmcnt 11:8 left at their maxima) that waits until at most n
// vector-memory operations of this wave are outstanding (n < 16).
template <bool CHAIN>
constexpr int refill_chunks() { return CHAIN ? 2 : 4; }
constexpr int wait_vm(int n) { return 0x0F70 | n; }

// With CHAIN the chain words move along: `fx`, `pool_ext`.
template <bool CHAIN>
__device__ void refill(Queue& q, int4& fe, int2& fx, int4* pool, int2* pool_ext, int64_t* pk,
                       int32_t* pi, int2* kb, int key_mode) {
  const int lane = lane_id();
  const int P = q.P;
  wave_mem_sync();   // this tick's pool appends are read below
  if (P <= kFront) {
    constexpr int NP = CHAIN ? 3 : 1;
    int4 e = make_int4(0, 0, 0, 0);
    int2 x = make_int2(0, 0);
    int64_t ck = kKeyMax;
    if (lane < P) {
      e = pool[lane];
      ck = composite(e.x, e.y);
      if constexpr (CHAIN) x = pool_ext[lane];
    }
    int32_t pay[NP];
    pay[0] = e.w;
    if constexpr (CHAIN) {
      pay[1] = x.x;
      pay[2] = x.y;
    }
    bitonic_sort64<NP>(ck, pay);
    const int32_t kk = comp_key(ck);
    fe = lane < P ? make_int4(kk, comp_id(ck), t_arr_of(kk, pay[0], key_mode), pay[0])
                  : make_int4(0, 0, 0, 0);
    if constexpr (CHAIN) fx = lane < P ? make_int2(pay[1], pay[2]) : make_int2(0, 0);
    q.fh = 0;
    q.fn = P;
    q.P = 0;
    return;
  }
  // Top-64 selection. `ck`/`idx` hold the 64 smallest keys seen so far,
  // ascending across lanes; thr is the largest of them. Later pool entries
  // below thr are collected in LDS and merged 64 at a time: a sorted batch,
  // reversed, taken elementwise-min with the best set gives a bitonic
  // sequence holding the 64 smallest of both, which one merge network sorts.
  const int4 e0 = pool[lane];
  int64_t ck = composite(e0.x, e0.y);
  int32_t idx[1] = {lane};
  bitonic_sort64<1>(ck, idx);
  int64_t thr = readlane64(ck, 63);
  int np = 0;   // candidates staged in pk/pi[0, np)
  auto flush = [&]() {
    int64_t bk = lane < np ? pk[lane] : kKeyMax;
    int32_t bi[1] = {lane < np ? pi[lane] : 0};
    bitonic_sort64<1>(bk, bi);
    const int64_t rk = shfl(bk, 63 - lane);
    const int32_t ri = shfl(bi[0], 63 - lane);
    if (rk < ck) { ck = rk; idx[0] = ri; }
    bitonic_merge64<1>(ck, idx);
    thr = readlane64(ck, 63);
    np = 0;
  };
  // The keys and ids of the remaining entries come into LDS through the LDS
  // DMA path (no registers held by loads in flight), kRefillChunks chunks of
  // 64 entries per round, double-buffered: the next round's loads are issued
  // before the current round is scanned. Lanes past the pool's end load its
  // last entry (an address in bounds) and are ignored.
  constexpr int G = refill_chunks<CHAIN>();
  int32_t* lk = reinterpret_cast<int32_t*>(kb);   // [2][G * kFront] keys
  int32_t* li = lk + 2 * G * kFront;              // [2][G * kFront] ids
  const int rounds = (P - kFront + G * kFront - 1) / (G * kFront);
  auto issue = [&](int r) {
    const int st = r & 1;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int i = kFront + (r * G + g) * kFront + lane;
      const int32_t* src = reinterpret_cast<const int32_t*>(pool + (i < P ? i : P - 1));
      __builtin_amdgcn_global_load_lds(src, (__attribute__((address_space(3))) void*)(lk + (st * G + g) * kFront),
                                       4, 0, 0);
      __builtin_amdgcn_global_load_lds(src + 1, (__attribute__((address_space(3))) void*)(li + (st * G + g) * kFront),
                                       4, 0, 0);
    }
  };
  issue(0);
  for (int r = 0; r < rounds; ++r) {
    // vector-memory counter: wait for this round's 2G loads, keep the next round's in flight
    if (r + 1 < rounds) {
      issue(r + 1);
      __builtin_amdgcn_s_waitcnt(wait_vm(2 * G));
    } else {
      __builtin_amdgcn_s_waitcnt(wait_vm(0));
    }
    const int st = r & 1;
#pragma unroll 1
    for (int g = 0; g < G; ++g) {
      const int i = kFront + (r * G + g) * kFront + lane;
      // Read through inline assembly: the compiler treats an LDS read after an
      // LDS DMA as dependent on every DMA in flight and would wait for the
      // next round's loads too; the explicit vmcnt wait above is the exact one.
      int32_t kv, iv;
      const uint32_t ak = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int32_t*)(lk + (st * G + g) * kFront + lane);
      const uint32_t ai = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) int32_t*)(li + (st * G + g) * kFront + lane);
      asm volatile("ds_read_b32 %0, %2\n\tds_read_b32 %1, %3\n\ts_waitcnt lgkmcnt(0)"
                   : "=v"(kv), "=v"(iv) : "v"(ak), "v"(ai));
      const int64_t kc = i < P ? composite(kv, iv) : kKeyMax;
      uint64_t cm = ballot(kc < thr);
      if (cm == 0) continue;
      if (np + popc64(cm) > kFront) {
        flush();
        cm = ballot(kc < thr);
        if (cm == 0) continue;
      }
      if ((cm >> lane) & 1ull) {
        const int pos = np + prefix_count(cm);
        pk[pos] = kc;
        pi[pos] = i;
      }
      np += popc64(cm);
    }
  }
  if (np > 0) flush();
  const int sel = idx[0];
  fe = pool[sel];
  if constexpr (CHAIN) fx = pool_ext[sel];
  // Compact the pool: selected entries below the new size are holes, filled
  // with the unselected entries of the last 64 positions (same count).
  const int Pn = P - kFront;
  const uint64_t tail_sel = wave_or(sel >= Pn ? (1ull << (sel - Pn)) : 0ull);
  const uint64_t fillers = ~tail_sel;
  const uint64_t holes = ballot(sel < Pn);
  int4 fill = make_int4(0, 0, 0, 0);
  int2 fillx = make_int2(0, 0);
  if (sel < Pn) {
    const int f = nth_set_bit(fillers, prefix_count(holes));
    fill = pool[Pn + f];
    if constexpr (CHAIN) fillx = pool_ext[Pn + f];
  }
  wave_mem_sync();
  if (sel < Pn) {
    pool[sel] = fill;
    if constexpr (CHAIN) pool_ext[sel] = fillx;
  }
  q.fh = 0;
  q.fn = kFront;
  q.P = Pn;
}

// Snapshot row entry of model m of env e from its state (one fp32 product
// per load statistic; validity byte). `part` selects which value to write
// (0..3: the four statistics, 4: validity), so lanes can share the work.
// The queue-depth statistic: recent dispatches / RPM limit for a blackbox
// model (Sec. 5.5), queue length / QCAP otherwise.
__device__ __forceinline__ float queue_stat(const SchedArgs& a, int32_t qlen, int32_t rpm,
                                            int32_t rcnt, float inv_rpm) {
  return rpm > 0 ? (float)rcnt * inv_rpm : (float)qlen * a.inv_qcap;
}

__device__ __forceinline__ void write_snap_part(const SchedArgs& a, int e, int m, int part,
                                                int32_t qlen, int32_t busy, int32_t ewma,
                                                int32_t backlog, int32_t cap, int32_t enabled,
                                                int32_t rpm, int32_t rcnt, float inv_rpm) {
  float* row = a.snap + (size_t)e * snap_stride(a.M);
  const int c = cap < 0 ? 0 : (cap > IM_MAX_SLOTS ? IM_MAX_SLOTS : cap);
  switch (part) {
    case 0: row[m] = queue_stat(a, qlen, rpm, rcnt, inv_rpm); break;
    case 1: row[a.M + m] = (float)busy * a.inv_tab[c]; break;
    case 2: row[2 * a.M + m] = (float)ewma * a.inv_lat; break;
    case 3: row[3 * a.M + m] = (float)backlog * a.inv_tab[IM_MAX_SLOTS + 1 + c]; break;
    case 4: {
      uint8_t* v = (uint8_t*)(row + snap_valid_offset(a.M));
      v[m] = (enabled != 0 && cap > 0 && qlen < a.qcap) ? 1 : 0;
      break;
    }
    default: break;
  }
}

__global__ void snapshot_kernel(SchedArgs a, int e0, int ne) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= (int64_t)ne * a.M) return;
  const int64_t em = (int64_t)e0 * a.M + i;
  const int e = (int)(em / a.M), m = (int)(em - (int64_t)e * a.M);
  const ModelRec r = a.ms[em];
  for (int part = 0; part < 5; ++part)
    write_snap_part(a, e, m, part, r.qlen, r.busy, r.ewma, r.backlog, r.cap, r.enabled,
                    r.rpm_limit, r.rpm_count, r.inv_rpm);
}

__device__ __forceinline__ int32_t wave_sum32(int32_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}

constexpr int kStageChunks = 4;   // arrival chunks (of 64) staged in LDS per round

// Per-model state of the env, one model per lane (lane m: model m) in
// registers for the whole tick.
struct LaneState {
  int32_t qlen, busy, ewma, backlog, fh, fn, P, busy_mask, next_done;
  int32_t rcnt;         // blackbox: dispatches in the window
  int32_t fmk, fmi;     // key and id of the front's last entry (its largest)
  int32_t chg;          // parts of the record that changed (CH_* bits)
};
enum { CH_STATS = 1, CH_FRONT = 2, CH_POOL = 4, CH_DONE = 8 };

__device__ __forceinline__ int32_t rl(int32_t v, int m) { return __builtin_amdgcn_readlane(v, m); }

// Per-model words of a wave's LDS scratch (one row of IM_MAX_MODELS each):
// sums over the lanes that work for a model, added with LDS atomics.
enum {
  MW_ACC = 0,    // newcomers admitted this round
  MW_SVC,        // their service time
  MW_CNT,        // rows of the current chunk routed to the model
  MW_KF,         // newcomers of the current chunk merged into the front
  MW_KP,         // newcomers of the current chunk appended to the pool
  MW_SEG,        // first lane of the model's segment in the current chunk
  MW_STARTED,    // slots filled this tick
  MW_WAIT,       // their waiting time
  MW_SVCOUT,     // their service time
  MW_DONE,       // completions
  MW_SLO,        // completions within budget
  MW_ND,         // earliest completion tick among the busy slots
  MW_NUM
};
enum { MD_LAT = 0, MD_COST, MD_NUM };   // 64-bit sums: latency, Q16 cost

// Adds v to a 64-bit counter without reading it back (a vector atomic whose
// result is unused: no wait, and integer sums do not depend on the order).
__device__ __forceinline__ void counter_add(int64_t* p, int64_t v) {
  atomicAdd(reinterpret_cast<unsigned long long*>(p), (unsigned long long)v);
}

// One wave per env. Every load that does not depend on the arrivals (the
// model records, one per lane, then each front's largest entry and blackbox
// window byte) is issued with the offsets; the env's rows are then loaded once
// (the first chunks stay in registers) and validated. 64 at a time they are
// partitioned by model (ballot + mbcnt ranks in id order give the tail-drop
// admission) and sorted once by (model, key, id) with a 64-lane bitonic
// network, so each model's newcomers form one sorted segment (a segmented
// sort), staged in LDS.
//
// Insertion works on every model of a chunk at once: a lane's newcomer goes
// to its model's front when it is below the front's largest entry (or the
// pool is empty and the front has room), else to the pool, whose position
// follows from a ballot over the lanes of its segment; one scattered store
// appends every model's pool-bound newcomers. Only models with front-bound
// newcomers then run a merge network, one model at a time (single-call pools
// load the fronts of two such models before merging either).
//
// Service is also model-parallel: lane (model, slot) fills its slot from the
// model's front (the head entries sit at known positions of the front array),
// advances it and completes it; per-model sums go through LDS atomics and the
// EWMA folds the completions in slot order. A model whose front runs dry is
// refilled from its pool on its own (rare), and its remaining slots then read
// the new front. Counters are added by lane (model, counter); records and
// the snapshot row are written once at the end, where they changed.
//
// RPM: the pool has (or had) a rate-limited model, so the blackbox dispatch
// windows are tracked; pools that never had one run without that code.
// CHAIN: multi-step chains (Sec. 4.3). The env's rows are its pending calls
// (spawned at the previous tick, in spawn order) then its arrivals; every
// call carries its query's two chain words through the queue, and a
// completion that is not its query's last call appends the next call, with
// the query's deadline, to the pending list of the next tick.
template <bool RPM, bool CHAIN, int PF>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(5, 8))) void schedule_kernel(SchedArgs a) {
  // sorted chunks; in the service phase the refill scan's key buffer, then
  // the counter staging
  __shared__ int4 stage[4][kStageChunks * 64];
  __shared__ int2 stage_x[4][CHAIN ? kStageChunks * 64 : 1];
  __shared__ int32_t hist_lds[4][IM_MAX_ACTIONS];
  __shared__ int32_t mw_lds[4][MW_NUM][IM_MAX_MODELS];
  __shared__ unsigned long long md_lds[4][MD_NUM][IM_MAX_MODELS];
  __shared__ int64_t pend_k[4][kFront];   // refill candidate staging
  __shared__ int32_t pend_i[4][kFront];
  static_assert(sizeof(int4) * kStageChunks * 64 >= sizeof(int2) * 2 * refill_chunks<CHAIN>() * kFront,
                "the refill buffer fits the stage");
  static_assert(kStageChunks * 64 >= (C_NUM / 2) * IM_MAX_MODELS, "the counter staging fits the stage");
  static_assert(IM_MAX_MODELS < 63, "model 63 marks rows not admitted");
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);   // wave-uniform
  const int e = (int)blockIdx.x * (int)(blockDim.x >> 6) + wv;   // 1, 2 or 4 envs per block
  if (e >= a.E) return;
  int4* st = stage[wv];
  int32_t* hist_s = hist_lds[wv];
  int32_t(*mw)[IM_MAX_MODELS] = mw_lds[wv];
  unsigned long long(*md)[IM_MAX_MODELS] = md_lds[wv];
  const int M = a.M, K = a.K, S = a.S;
  // a / K for actions a < 64 as a multiply-high by ceil(2^32 / K) (exact for a < 2^32 / K)
  const uint32_t kmag = K == 1 ? 0u : 0xffffffffu / (uint32_t)K + 1u;
  // bits of a model index (M <= 32)
  const int mbits = M <= 1 ? 0 : 32 - __builtin_clz((uint32_t)(M - 1));
  const size_t em0 = (size_t)e * M;
  ModelRec* recs = a.ms + em0;
  const bool ml = lane < M;   // this lane holds model `lane`

  // ---- first loads, issued together: the model records (lane m: model m;
  // the other lanes read model M - 1's and clear theirs once the rows' loads
  // are issued) and the env's CSR offsets (scalar loads, so waiting for them
  // does not wait for the records) ----
  const int4* rp = reinterpret_cast<const int4*>(recs + (ml ? lane : M - 1));
  int4 r0 = rp[0], r1 = rp[1], r2 = rp[2], r3 = rp[3];
  const int32_t lo = load_uniform(a.offsets + e), hi = load_uniform(a.offsets + e + 1);
  int32_t abase = lo;
  if constexpr (CHAIN) abase = load_uniform(a.roff + e);   // the rows' outputs start at roff[e]
  int32_t bad = 0;
  if (lo < 0 || hi < lo || hi > a.n_total || hi - lo > a.max_arrivals) bad = IM_ERR_COUNT;
  if (CHAIN && load_uniform(a.csr_bad) != 0) bad = IM_ERR_COUNT;   // the rows build found no usable arrival
  const int32_t n = bad ? 0 : hi - lo;   // arrivals

  // ---- the env's rows: the first chunks are loaded (and kept) before
  // anything waits for them, then validated ----
  // Row r of the env is a pending call (r < pc, chain pools: valid by
  // construction; its budget is what is left of its query's) or arrival
  // lo + r - pc. Single-call pools need only the offsets to load their rows,
  // so those loads are in flight with the records.
  constexpr int kKeep = 2;                            // chunks kept in registers
  int32_t c_ac[kKeep], c_qi[kKeep], c_bu[kKeep], c_sv[kKeep], c_ro[kKeep];
#pragma unroll
  for (int c = 0; c < kKeep; ++c) {
    c_ac[c] = -1;
    c_qi[c] = 0;
    c_bu[c] = 1;
    c_sv[c] = 1;
    c_ro[c] = 0;
  }
  auto load_arrival = [&](int32_t r, int32_t i, int32_t& ac, int32_t& qi, int32_t& bu, int32_t& sv, int32_t& ro) {
    ac = a.actions[abase + r];
    qi = a.q_idx[i];
    bu = a.budget[i];
    sv = a.base_svc[i];
    if (a.role) ro = a.role[i];
  };
  if constexpr (!CHAIN) {
#pragma unroll
    for (int c = 0; c < kKeep; ++c) {
      const int32_t r = c * 64 + lane;
      if (r < n) load_arrival(r, lo + r, c_ac[c], c_qi[c], c_bu[c], c_sv[c], c_ro[c]);
    }
  }
  if (!ml) {
    r0 = make_int4(0, 0, 0, 0);
    r1 = r0;
    r2 = r0;
    r3 = r0;
  }
  // The tick and the next request id live in the env's first record in
  // device memory, so a captured sequence of ticks replays with the right time.
  const int32_t next_id = rl(r2.y, 0);
  const int32_t t = rl(r2.z, 0);
  // chain pools: this tick's pending calls (buffer of parity t) and the next
  // tick's (parity t + 1)
  const int4* pend_cur = nullptr;
  int4* pend_nxt = nullptr;
  int32_t pc = 0;
  if constexpr (CHAIN) {
    const size_t E = (size_t)a.E;
    pend_cur = a.pend + ((size_t)(t & 1) * E + e) * a.pend_cap;
    pend_nxt = a.pend + ((size_t)((t + 1) & 1) * E + e) * a.pend_cap;
    pc = a.pcnt[(size_t)(t & 1) * E + e];
  }
  const int32_t nrows = pc + n;          // rows: pending calls, then arrivals

  int32_t c_bs[kKeep];                                // budget << 16 | base_svc (16 bits each)
  int32_t c_xa[kKeep], c_xb[kKeep];                   // chain words (chain pools)
#pragma unroll
  for (int c = 0; c < kKeep; ++c) {
    c_bs[c] = 0;
    c_xa[c] = 0;
    c_xb[c] = 0;
  }
  int32_t berr = 0;
  // validation of an arrival, its packed service/budget word and (chain
  // pools) its chain words
  auto check_arrival = [&](int32_t i, int32_t ac, int32_t qi, int32_t bu, int32_t sv, int32_t ro, int32_t& bs,
                           int32_t& xa, int32_t& xb) {
    if (ac < -1 || ac >= a.A) berr |= IM_ERR_ACTION;
    if (qi < 0 || (int64_t)qi >= a.Q) berr |= IM_ERR_QIDX;
    if (a.role && (ro < 0 || ro >= a.n_roles)) berr |= IM_ERR_ROLE;
    if (bu < 1) berr |= IM_ERR_BUDGET;
    if (sv < 1 || sv > IM_SVC_MAX) berr |= IM_ERR_SVC;
    if (CHAIN) {
      const int32_t ns = a.n_steps[i];
      if (ns < 1 || ns > a.max_steps) berr |= IM_ERR_STEPS;
      xa = chain_a(qi, 0, ns);
      xb = chain_b(sv, bu, ro);
    }
    bs = (int32_t)(((uint32_t)bu << 16) | ((uint32_t)sv & 0xffffu));
  };
  // row r of a chain pool's env, loaded and validated
  auto load_row = [&](int32_t r, int32_t& ac, int32_t& bs, int32_t& xa, int32_t& xb) {
    if (CHAIN && r < pc) {
      ac = a.actions[abase + r];
      if (ac < -1 || ac >= a.A) berr |= IM_ERR_ACTION;
      const int4 pr = pend_cur[r];
      const int32_t bu = remaining_budget(pr.z, t);
      xa = pr.x;
      xb = pr.y;
      bs = (int32_t)(((uint32_t)bu << 16) | ((uint32_t)chain_base(pr.y) & 0xffffu));
      return;
    }
    const int32_t i = lo + (r - pc);
    int32_t qi = 0, bu = 1, sv = 1, ro = 0;
    load_arrival(r, i, ac, qi, bu, sv, ro);
    check_arrival(i, ac, qi, bu, sv, ro, bs, xa, xb);
  };
#pragma unroll
  for (int c = 0; c < kKeep; ++c) {
    const int32_t r = c * 64 + lane;
    if (r < nrows) {
      if constexpr (CHAIN) {
        load_row(r, c_ac[c], c_bs[c], c_xa[c], c_xb[c]);
      } else {
        check_arrival(lo + r, c_ac[c], c_qi[c], c_bu[c], c_sv[c], c_ro[c], c_bs[c], c_xa[c], c_xb[c]);
      }
    }
  }
  for (int32_t base = kKeep * 64; base < nrows; base += 64) {
    const int32_t r = base + lane;
    int32_t ac, bs, xa, xb;
    if (r < nrows) load_row(r, ac, bs, xa, xb);
  }
  if (nrows > 0) {
    // wave-wide OR of the error bits, one ballot each
    if (ballot(berr & IM_ERR_QIDX)) bad |= IM_ERR_QIDX;
    if (ballot(berr & IM_ERR_BUDGET)) bad |= IM_ERR_BUDGET;
    if (ballot(berr & IM_ERR_SVC)) bad |= IM_ERR_SVC;
    if (ballot(berr & IM_ERR_ACTION)) bad |= IM_ERR_ACTION;
    if (a.role && ballot(berr & IM_ERR_ROLE)) bad |= IM_ERR_ROLE;
    if (CHAIN && ballot(berr & IM_ERR_STEPS)) bad |= IM_ERR_STEPS;
  }
  // Each front's largest entry (needed when newcomers arrive while the pool is
  // not empty or the front is full) and the blackbox window byte leaving at
  // this tick: issued once the rows are validated (a
  // wait for them would otherwise wait for these too), in flight while they
  // are sorted.
  int32_t fmk = 0, fmi = 0, rold_l = 0;
  if (ml && r1.w > 0 && (r2.x > 0 || r1.w == kFront)) {
    const int2 f = *reinterpret_cast<const int2*>(a.front + (em0 + lane) * kFront + r1.z + r1.w - 1);
    fmk = f.x;
    fmi = f.y;
  }
  // lane m: the reciprocals its snapshot statistics are multiplied by,
  // 1/max(c_m,1) and 1/(max(c_m,1) budget_max) (c_m is not changed by a tick)
  float inv_busy_l = 0.f, inv_back_l = 0.f;
  if (ml) {
    const int c = r1.x < 0 ? 0 : (r1.x > IM_MAX_SLOTS ? IM_MAX_SLOTS : r1.x);
    inv_busy_l = a.inv_tab[c];
    inv_back_l = a.inv_tab[IM_MAX_SLOTS + 1 + c];
  }
  const int32_t rpm_l = RPM && ml ? r3.y : 0;   // lane m: model m's limit (0: not a blackbox model)
  const bool track_l = RPM && ml && (rpm_l > 0 || r3.z > 0);
  if (track_l) rold_l = a.rpm_ring[(em0 + lane) * kRpmRing + (t % kRpmWindow)];

  LaneState L;
  L.qlen = r0.x; L.busy = r0.y; L.ewma = r0.z; L.backlog = r0.w;
  L.fh = r1.z; L.fn = r1.w;
  L.P = r2.x; L.busy_mask = r2.w; L.next_done = r3.x;
  L.rcnt = RPM ? r3.z : 0;
  L.fmk = fmk; L.fmi = fmi;
  L.chg = 0;
  const int32_t cap_l = r1.x, en_l = r1.y;
  const int32_t inv_rpm_bits = RPM ? r3.w : 0;
  if (bad) {
    // The env's state is untouched and time still advances: busy slots keep
    // their remaining service, so their completion ticks move one tick later.
    if (lane == 0) {
      atomicOr(a.err, bad);
      recs[0].t = t + 1;
    }
    for (int m = 0; m < M; ++m) {
      if (rl(L.busy_mask, m) == 0) continue;
      int4* sl = a.slots + (em0 + m) * S;
      if (lane < S) {
        int4 v = sl[lane];
        if (v.x >= 0) {
          v.z += 1;
          sl[lane] = v;
        }
      }
    }
    if (ml && L.busy_mask != 0) recs[lane].next_done = L.next_done + 1;
    if constexpr (CHAIN) {
      // the env's pending calls stay pending
      for (int i = lane; i < pc; i += 64) pend_nxt[i] = pend_cur[i];
      if (lane == 0) a.pcnt[(size_t)((t + 1) & 1) * a.E + e] = pc;
    }
    // a tracked window still slides: the dispatches of tick t - 60 leave it
    if (RPM && track_l && rold_l != 0) {
      a.rpm_ring[(em0 + lane) * kRpmRing + (t % kRpmWindow)] = 0;
      recs[lane].rpm_count = L.rcnt - rold_l;
      a.snap[(size_t)e * snap_stride(M) + lane] = queue_stat(a, L.qlen, rpm_l, L.rcnt - rold_l, __int_as_float(inv_rpm_bits));
    }
    return;
  }

  hist_s[lane] = 0;                     // IM_MAX_ACTIONS == 64 lanes
  if (lane < IM_MAX_MODELS) {
    mw[MW_ACC][lane] = 0;
    mw[MW_SVC][lane] = 0;
  }
  // lane m < M: room left in model m's queue at the snapshot
  const int32_t room_l = ml ? a.qcap - L.qlen : 0;
  int32_t prior_l = 0;      // lane m: requests routed to model m so far (id order)
  int32_t acc_l = 0;        // lane m: requests accepted by model m so far
  int32_t nomodel = 0;
  const int n_chunks = (nrows + 63) / 64;
  int32_t pn = 0;            // pending calls spawned for the next tick
  int32_t q_done = 0, q_met = 0;
  uint64_t wrote = 0;        // models whose front array was written this tick
  int2* stx = stage_x[wv];
  const int rounds = n_chunks > 0 ? (n_chunks + kStageChunks - 1) / kStageChunks : 1;

  for (int r = 0; r < rounds; ++r) {
    const int c0 = r * kStageChunks;
    const int nch = n_chunks - c0 < kStageChunks ? n_chunks - c0 : kStageChunks;
    // ---- partition, admission and one sort per chunk ----
#pragma unroll
    for (int c = 0; c < kStageChunks; ++c) {
      if (c >= nch) break;
      const int32_t base = (c0 + c) * 64;
      const int32_t i = base + lane;   // row of the env
      const bool in = i < nrows;
      int32_t ac = c < kKeep ? c_ac[c < kKeep ? c : 0] : -1;
      int32_t bs = c < kKeep ? c_bs[c < kKeep ? c : 0] : 0;
      int32_t xa = c < kKeep ? c_xa[c < kKeep ? c : 0] : 0;
      int32_t xb = c < kKeep ? c_xb[c < kKeep ? c : 0] : 0;
      if (r != 0 || c >= kKeep) {
        ac = -1;
        bs = 0;
        if (in) load_row(i, ac, bs, xa, xb);
      }
      const int32_t bu = bs >> 16, sv = bs & 0xffff;
      const int32_t mdl = ac < 0 ? -1 : (K == 1 ? ac : (int32_t)__umulhi((uint32_t)ac, kmag));
      nomodel += popc64(ballot(in && ac < 0));
      if (in && ac >= 0) atomicAdd(&hist_s[ac], 1);   // routed requests per action
      // The lanes routed to this row's model: one ballot per bit of the
      // model index. A row's rank among its model's rows in id order is the
      // model's count before this chunk plus its lanes below; the first lane
      // of each model passes the chunk's count to the model's lane.
      const bool routed = in && mdl >= 0;
      uint64_t same = ballot(routed);
      for (int b = 0; b < mbits; ++b) {
        const bool bit = ((mdl >> b) & 1) != 0;
        const uint64_t bb = ballot(routed && bit);
        same &= bit ? bb : ~bb;
      }
      const int msrc = mdl >= 0 ? mdl : 0;
      const int below = prefix_count(same);
      const int32_t rank = shfl(prior_l, msrc) + below;
      if (ml) mw[MW_CNT][lane] = 0;
      if (routed && below == 0) mw[MW_CNT][mdl] = popc64(same);
      if (ml) prior_l += mw[MW_CNT][lane];
      const int32_t room = shfl(room_l, msrc);
      const bool acc = in && mdl >= 0 && rank < room;
      const int32_t d = ac - mdl * K;
      const int32_t svc = sv * (d + 1);
      if (acc) {                                     // admitted count and service time per model
        atomicAdd(&mw[MW_ACC][mdl], 1);
        atomicAdd(&mw[MW_SVC][mdl], svc);
      }
      // Sort key (32 bits): model (63 for rows not admitted) | key - t biased by
      // 2^17 | lane. Every row of the chunk enters at t, so ordering by key - t
      // is ordering by key; with budget in [-32768, 32767] (a later call of a
      // chain may be past its deadline) and svc in [1, 65520], key - t lies in
      // [-98288, 32767] (18 bits once biased). The lane keeps ties in id order
      // and locates the row's packed service/budget word.
      const int32_t rk = a.key_mode == IM_KEY_DEADLINE ? bu : (a.key_mode == IM_KEY_FCFS ? 0 : bu - svc);
      uint32_t sk = ((uint32_t)(acc ? mdl : 63) << 24) | (((uint32_t)(rk + 131072) & 0x3ffffu) << 6) |
                    (uint32_t)lane;
      const int32_t pay = (int32_t)(((uint32_t)svc & 0xffffu) | ((uint32_t)bu << 16));
      // Rows of the chunk sit in its first lanes: sort only the smallest power
      // of two of lanes holding them (the other lanes hold rows of model 63).
      // When at most a quarter of them are admitted (full queues drop the
      // rest), the admitted rows' keys are first moved to the lowest lanes, in
      // lane order, and only those are sorted; every key keeps its row's lane.
      const int nr = nrows - base < 64 ? nrows - base : 64;
      const uint64_t am = ballot(acc);
      const int na = popc64(am);
      if (4 * na <= nr) {
        const int pos = acc ? prefix_count(am) : na + prefix_count(~am);
        sk = (uint32_t)__builtin_amdgcn_ds_permute(pos * 4, (int32_t)sk);
        if (na > 1) bitonic_sort_first(sk, na);
      } else {
        bitonic_sort_first(sk, nr);
      }
      const int src = (int)(sk & 63u);
      const int32_t skey = t + (int32_t)((sk >> 6) & 0x3ffffu) - 131072;
      const int32_t sid = next_id + base + src;
      st[c * 64 + lane] = make_int4(skey, sid, shfl(pay, src), (int32_t)(sk >> 24));
      if constexpr (CHAIN) stx[c * 64 + lane] = make_int2(shfl(xa, src), shfl(xb, src));
    }
    const bool last = r == rounds - 1;

    // lane m: newcomers admitted by model m this round and their service time
    if (lane < IM_MAX_MODELS) {
      const int32_t k_round = mw[MW_ACC][lane], svc_round = mw[MW_SVC][lane];
      mw[MW_ACC][lane] = 0;   // LDS accesses of one wave stay in order
      mw[MW_SVC][lane] = 0;
      if (ml && k_round > 0) {
        L.qlen += k_round;
        L.backlog += svc_round;
        acc_l += k_round;
        L.chg |= CH_STATS;
      }
    }

    // ---- insertion, every model of a chunk at once ----
    for (int c = 0; c < nch; ++c) {
      const int4 en = st[c * 64 + lane];
      const int mdl = en.w;                  // 63: not admitted (sorted last)
      const bool in = mdl < M;
      if (ballot(in) == 0) continue;
      const int src = in ? mdl : 0;
      const int32_t Pm = shfl(L.P, src), fnm = shfl(L.fn, src);
      const int64_t fm = composite(shfl(L.fmk, src), shfl(L.fmi, src));
      const int64_t cp = composite(en.x, en.y);
      // front-bound: below the front's largest entry, or the pool is empty and
      // the front has room (every front key stays below every pool key)
      const bool fb = in && ((Pm == 0 && fnm < kFront) || (fnm > 0 && cp < fm));
      const bool pb = in && !fb;
      const int prv = shfl(mdl, (lane + 63) & 63);
      const int nxt = shfl(mdl, (lane + 1) & 63);
      const uint64_t heads = ballot(in && (lane == 0 || prv != mdl));
      const uint64_t upto = lane == 63 ? ~0ull : ((2ull << lane) - 1ull);   // lanes <= this one
      const int seg = in ? 63 - __builtin_clzll((heads & upto) | 1ull) : 0;        // the segment's first lane
      const uint64_t below_seg = (1ull << seg) - 1ull;
      const uint64_t pbm = ballot(pb), fbm = ballot(fb);
      if (pb) {
        // position among the segment's pool-bound newcomers (a suffix of it)
        const int o = prefix_count(pbm) - popc64(pbm & below_seg);
        const size_t pos = (em0 + mdl) * a.qcap + Pm + o;
        a.pool[pos] = make_int4(en.x, en.y, t, en.z);
        if constexpr (CHAIN) a.pool_ext[pos] = stx[c * 64 + lane];
      }
      if (ml) {
        mw[MW_KF][lane] = 0;
        mw[MW_KP][lane] = 0;
      }
      if (in && (lane == 63 || nxt != mdl)) {   // the segment's last lane
        const uint64_t segm = upto & ~below_seg;
        mw[MW_KF][mdl] = popc64(fbm & segm);
        mw[MW_KP][mdl] = popc64(pbm & segm);
        mw[MW_SEG][mdl] = seg;
      }
      const int32_t kf_l = ml ? mw[MW_KF][lane] : 0;
      const int32_t kp_l = ml ? mw[MW_KP][lane] : 0;
      if (kp_l > 0) {
        L.P += kp_l;
        L.chg |= CH_POOL;
      }
      // models with front-bound newcomers: merge them into the front
      uint64_t merges = ballot(kf_l > 0);
      if constexpr (PF == 1) {
        while (merges) {
          const int m = __builtin_ctzll(merges);
          merges &= merges - 1;
          const size_t em = em0 + m;
          Queue q;
          q.fh = rl(L.fh, m);
          q.fn = rl(L.fn, m);
          q.P = rl(L.P, m);
          const int lim = rl(kf_l, m);
          const int s0 = __builtin_amdgcn_readfirstlane(mw[MW_SEG][m]);
          if ((wrote >> m) & 1ull) wave_mem_sync();   // this model's front was written this tick
          int4 fe = make_int4(0, 0, 0, 0);
          int2 fx = make_int2(0, 0);
          if (lane < q.fn) {
            fe = a.front[em * kFront + q.fh + lane];   // fh + fn <= kFront
            if constexpr (CHAIN) fx = a.front_ext[em * kFront + q.fh + lane];
          }
          const int32_t okey = fe.x, oid = fe.y;
          const int ofh = q.fh, ofn = q.fn;
          merge_front<CHAIN>(q, fe, fx, st + c * 64 + s0, stx + c * 64 + s0, lim, a.key_mode,
                             a.pool + em * a.qcap, CHAIN ? a.pool_ext + em * a.qcap : nullptr);
          // the front now starts at 0; entries that kept their position are not rewritten
          const bool same = ofh == 0 && lane < ofn && okey == fe.x && oid == fe.y;
          if (lane < q.fn && !same) {
            a.front[em * kFront + lane] = fe;
            if constexpr (CHAIN) a.front_ext[em * kFront + lane] = fx;
          }
          wrote |= 1ull << m;
          const int32_t nk = rl(fe.x, q.fn - 1), ni = rl(fe.y, q.fn - 1);   // q.fn >= 1 after a merge
          if (lane == m) {
            L.fh = 0;
            L.fn = q.fn;
            L.P = q.P;
            L.fmk = nk;
            L.fmi = ni;
            L.chg |= CH_FRONT | CH_POOL;
          }
        }
      } else {
        // PF models at a time, whose fronts are loaded together (one round trip
        // per group instead of one per model); each is merged by the same
        // steps as in the loop above (two copies: sharing them through one
        // inlined helper costs the one-model kernels registers)
        while (merges) {
          int gm[PF];
          uint64_t gmask = 0;
  #pragma unroll
          for (int d = 0; d < PF; ++d) {
            gm[d] = merges ? __builtin_ctzll(merges) : -1;
            if (gm[d] >= 0) gmask |= 1ull << gm[d];
            merges &= merges - 1;
          }
          if (wrote & gmask) wave_mem_sync();   // a front written earlier this tick is read below
          int4 pfe[PF];
          int2 pfx[PF];
  #pragma unroll
          for (int d = 0; d < PF; ++d) {
            pfe[d] = make_int4(0, 0, 0, 0);
            pfx[d] = make_int2(0, 0);
            if (gm[d] >= 0) {
              const int fh = rl(L.fh, gm[d]), fn = rl(L.fn, gm[d]);
              if (lane < fn) {
                pfe[d] = a.front[(em0 + gm[d]) * kFront + fh + lane];
                if constexpr (CHAIN) pfx[d] = a.front_ext[(em0 + gm[d]) * kFront + fh + lane];
              }
            }
          }
  #pragma unroll
          for (int d = 0; d < PF; ++d) {
            const int m = gm[d];
            if (m < 0) break;
            const size_t em = em0 + m;
            Queue q;
            q.fh = rl(L.fh, m);
            q.fn = rl(L.fn, m);
            q.P = rl(L.P, m);
            const int lim = rl(kf_l, m);
            const int s0 = __builtin_amdgcn_readfirstlane(mw[MW_SEG][m]);
            int4 fe = pfe[d];
            int2 fx = pfx[d];
            const int32_t okey = fe.x, oid = fe.y;
            const int ofh = q.fh, ofn = q.fn;
            merge_front<CHAIN>(q, fe, fx, st + c * 64 + s0, stx + c * 64 + s0, lim, a.key_mode,
                               a.pool + em * a.qcap, CHAIN ? a.pool_ext + em * a.qcap : nullptr);
            // the front now starts at 0; entries that kept their position are not rewritten
            const bool same = ofh == 0 && lane < ofn && okey == fe.x && oid == fe.y;
            if (lane < q.fn && !same) {
              a.front[em * kFront + lane] = fe;
              if constexpr (CHAIN) a.front_ext[em * kFront + lane] = fx;
            }
            wrote |= 1ull << m;
            const int32_t nk = rl(fe.x, q.fn - 1), ni = rl(fe.y, q.fn - 1);   // q.fn >= 1 after a merge
            if (lane == m) {
              L.fh = 0;
              L.fn = q.fn;
              L.P = q.P;
              L.fmk = nk;
              L.fmi = ni;
              L.chg |= CH_FRONT | CH_POOL;
            }
          }
        }
      }
    }
    if (!last) continue;

    // ---- service: fill free slots below c_m from the queue head, then one
    // tick of service (every model at once: lane = (model, slot)) ----
    // A blackbox model dispatches only while its window (ticks t-59..t)
    // holds fewer than rpm dispatches (App. C): the rest wait in the queue.
    const int capc_l = cap_l < 0 ? 0 : (cap_l > S ? S : cap_l);
    const uint32_t free_l = ml ? (~(uint32_t)L.busy_mask & ((1u << capc_l) - 1u)) : 0u;
    const int32_t window_l = L.rcnt - rold_l;
    int32_t npop_l = min((int32_t)__popc(free_l), L.qlen);
    if (RPM && rpm_l > 0) npop_l = min(npop_l, rpm_l > window_l ? rpm_l - window_l : 0);
    const bool due_l = ml && L.busy_mask != 0 && L.next_done <= t;
    const uint64_t serve = ballot(npop_l > 0 || due_l);
    if (ml) {
      mw[MW_STARTED][lane] = 0;
      mw[MW_WAIT][lane] = 0;
      mw[MW_SVCOUT][lane] = 0;
      mw[MW_DONE][lane] = 0;
      mw[MW_SLO][lane] = 0;
      mw[MW_ND][lane] = 0x7fffffff;
      md[MD_LAT][lane] = 0;
      md[MD_COST][lane] = 0;
    }
    // Fronts that run dry this tick (rare): the remaining front entries stay
    // at the head and the smallest pool entries follow them (a top-64
    // selection over the pool); what does not fit goes back to the pool.
    uint64_t dry = ballot(npop_l > L.fn);
    if (dry != 0) {
      if (dry & wrote) wave_mem_sync();
      while (dry) {
        const int m = __builtin_ctzll(dry);
        dry &= dry - 1;
        const size_t em = em0 + m;
        const int ofh = rl(L.fh, m), ofn = rl(L.fn, m);
        int4 old = make_int4(0, 0, 0, 0);
        int2 oldx = make_int2(0, 0);
        if (lane < ofn) {
          old = a.front[em * kFront + ofh + lane];
          if constexpr (CHAIN) oldx = a.front_ext[em * kFront + ofh + lane];
        }
        Queue q;
        q.P = rl(L.P, m);
        q.fh = 0;
        q.fn = 0;
        int4 fe;
        int2 fx;
        int4* pool = a.pool + em * a.qcap;
        int2* pool_x = CHAIN ? a.pool_ext + em * a.qcap : nullptr;
        refill<CHAIN>(q, fe, fx, pool, pool_x, pend_k[wv], pend_i[wv], reinterpret_cast<int2*>(st), a.key_mode);
        const int nsel = q.fn;                                   // >= 1: P > 0
        const int nf = ofn + nsel < kFront ? ofn + nsel : kFront;
        const int back = ofn + nsel - nf;                        // largest selected entries returned
        if (lane >= nsel - back && lane < nsel) {
          pool[q.P + lane - (nsel - back)] = fe;
          if constexpr (CHAIN) pool_x[q.P + lane - (nsel - back)] = fx;
        }
        q.P += back;
        const int sh = (lane - ofn) & 63;
        const int4 se = make_int4(shfl(fe.x, sh), shfl(fe.y, sh), shfl(fe.z, sh), shfl(fe.w, sh));
        const int4 ne = lane < ofn ? old : se;
        int2 nx = oldx;
        if constexpr (CHAIN) {
          const int2 sx2 = make_int2(shfl(fx.x, sh), shfl(fx.y, sh));
          nx = lane < ofn ? oldx : sx2;
        }
        if (lane < nf) {
          a.front[em * kFront + lane] = ne;
          if constexpr (CHAIN) a.front_ext[em * kFront + lane] = nx;
        }
        const int32_t nk = rl(ne.x, nf - 1), ni = rl(ne.y, nf - 1);
        if (lane == m) {
          L.P = q.P;
          L.fh = 0;
          L.fn = nf;
          L.fmk = nk;
          L.fmi = ni;
          L.chg |= CH_FRONT | CH_POOL;
        }
        wrote |= 1ull << m;
      }
      wave_mem_sync();
    }
    if (serve != 0) {
      if (serve & wrote) wave_mem_sync();   // fronts written this tick are read below
      const int mpp = kWave / S;             // models per pass
      const int mi = lane / S, s = lane - mi * S;
      for (int m0 = 0; m0 < M; m0 += mpp) {
        const uint64_t pass = (mpp >= 64 ? ~0ull : ((1ull << mpp) - 1ull)) << m0;
        if ((serve & pass) == 0) continue;
        const int m = m0 + mi;
        const bool sv = mi < mpp && m < M && ((serve >> m) & 1ull);   // lane serves slot s of model m
        const int ms = sv ? m : 0;
        const size_t em = em0 + ms;
        const uint32_t fr = (uint32_t)shfl((int32_t)free_l, ms);
        const int32_t np = shfl(npop_l, ms), fhm = shfl(L.fh, ms);
        // slot: {id, t_arr, tick of completion, budget}; id -1 = empty
        int4 sl = make_int4(-1, 0, 0, 0);
        int2 sx = make_int2(0, 0);
        if (sv) {
          sl = a.slots[em * S + s];
          if constexpr (CHAIN) sx = a.slot_ext[em * S + s];
        }
        // free slots are filled in slot order from the front's head
        const int rank = __popc(fr & ((1u << s) - 1u));
        const bool pop = sv && ((fr >> s) & 1u) && rank < np;
        if (pop) {
          const int4 pe = a.front[em * kFront + fhm + rank];
          if constexpr (CHAIN) sx = a.front_ext[em * kFront + fhm + rank];
          const int32_t svc = pe.w & 0xffff;
          sl = make_int4(pe.y, pe.z, t + svc - 1, pe.w >> 16);   // budget signed
          atomicAdd(&mw[MW_STARTED][m], 1);
          atomicAdd(&mw[MW_WAIT][m], t - pe.z);
          atomicAdd(&mw[MW_SVCOUT][m], svc);
        }
        // ---- one tick of service; a slot filled at t with svc = 1 completes at t ----
        const bool busy_slot = sv && sl.x >= 0;
        const bool done = busy_slot && sl.z <= t;   // == t in every valid state
        const int32_t lat = t - sl.y + 1;
        if (done) {
          // cost latency / budget of Eq. 2 in Q16 (budget >= 1); beta: the
          // query's budget (chains; the call's own for single steps)
          const uint32_t bud = CHAIN ? (uint32_t)chain_beta(sx.y) : (uint32_t)sl.w;
          uint64_t cq = (uint64_t)(((uint32_t)lat << 16) / bud);   // latency < 2^16
          if (lat >= 65536) cq = ((uint64_t)(uint32_t)lat << 16) / bud;
          atomicAdd(&mw[MW_DONE][m], 1);
          if (lat <= sl.w) atomicAdd(&mw[MW_SLO][m], 1);
          atomicAdd(&md[MD_LAT][m], (unsigned long long)(int64_t)lat);
          atomicAdd(&md[MD_COST][m], (unsigned long long)cq);
        }
        if constexpr (CHAIN) {
          // call k + 1 of the query, for the next tick, with the query's deadline
          // (spawn order: models in order, then slots, which is lane order)
          const bool more = done && chain_k(sx.x) + 1 < chain_n(sx.x);
          const uint64_t spawn = ballot(more);
          if (more) pend_nxt[pn + prefix_count(spawn)] = make_int4(sx.x + (1 << 24), sx.y, sl.y + sl.w, 0);
          pn += popc64(spawn);
          const bool fin = done && !more;
          q_done += popc64(ballot(fin));
          q_met += popc64(ballot(fin && lat <= sl.w));
        }
        if (busy_slot && !done) atomicMin(&mw[MW_ND][m], sl.z);
        if (pop || done) {
          if (done) sl = make_int4(-1, 0, 0, 0);
          a.slots[em * S + s] = sl;
          if constexpr (CHAIN) a.slot_ext[em * S + s] = sx;
        }
        const uint64_t bm = ballot(busy_slot && !done);
        // lane m of this pass: its busy slots and the EWMA over its
        // completions in slot order (alpha = 1/8, Q8, floor)
        const int32_t latd = done ? lat : 0;
        const bool mine = ml && (((pass & serve) >> lane) & 1ull);
        const int base_l = mine ? (lane - m0) * S : 0;
        int32_t ew = L.ewma;
        for (int s2 = 0; s2 < S; ++s2) {
          const int32_t ls = shfl(latd, base_l + s2);
          if (mine && ls > 0) {
            const int64_t delta = (int64_t)ls * 256 - ew;
            const int64_t stepv = delta >= 0 ? (delta >> 3) : -((-delta + 7) >> 3);
            ew = (int32_t)(ew + stepv);
          }
        }
        if (mine) {
          L.ewma = ew;
          L.busy_mask = (int32_t)((bm >> base_l) & ((1ull << S) - 1ull));
        }
      }
      // lane m: the model's queue after its pops
      if (ml && ((serve >> lane) & 1ull)) {
        L.qlen -= npop_l;
        L.backlog -= mw[MW_SVCOUT][lane];
        L.busy = __popc((uint32_t)L.busy_mask);
        L.next_done = mw[MW_ND][lane];
        L.fh += npop_l;
        L.fn -= npop_l;
        L.chg |= CH_STATS | CH_POOL | CH_DONE | (npop_l > 0 ? CH_FRONT : 0);
      }
    }
    if constexpr (RPM) {
      // this tick's recorded dispatches enter the window; those of tick t - 60 leave it
      const int32_t rec = rpm_l > 0 ? mw[MW_STARTED][lane] : 0;
      if (track_l && rec != rold_l) a.rpm_ring[(em0 + lane) * kRpmRing + (t % kRpmWindow)] = (uint8_t)rec;
      if (ml && window_l + rec != L.rcnt) {
        L.rcnt = window_l + rec;
        L.chg |= CH_STATS | CH_DONE;
      }
    }
  }

  // ---- counters, by lane (model, counter); service sums from LDS ----
  {
    const uint64_t act = ballot(ml && (prior_l != 0 || mw[MW_STARTED][lane] != 0 || mw[MW_DONE][lane] != 0));
    static_assert(C_NUM == 8, "eight counters per model");
    for (int m0 = 0; m0 < M; m0 += 8) {
      if (((act >> m0) & 0xffull) == 0) continue;
      const int m = m0 + (lane >> 3), c = lane & 7;
      const int ms = m < M ? m : 0;
      const int32_t pr = shfl(prior_l, ms), ac = shfl(acc_l, ms);
      if (m < M && ((act >> m) & 1ull)) {
        int64_t x;
        switch (c) {
          case C_REJ_OVERFLOW: x = pr - ac; break;
          case C_ENQUEUED: x = ac; break;
          case C_STARTED: x = mw[MW_STARTED][m]; break;
          case C_COMPLETED: x = mw[MW_DONE][m]; break;
          case C_SLO_MET: x = mw[MW_SLO][m]; break;
          case C_LAT_SUM: x = (int64_t)md[MD_LAT][m]; break;
          case C_WAIT_SUM: x = mw[MW_WAIT][m]; break;
          default: x = (int64_t)md[MD_COST][m]; break;
        }
        if (x != 0) counter_add(a.cnt + (em0 + m) * C_NUM + c, x);
      }
    }
  }

  // ---- records of the models whose state changed (lane m: model m) ----
  if (ml) {
    int4* rp = reinterpret_cast<int4*>(recs + lane);
    if (L.chg & CH_STATS) rp[0] = make_int4(L.qlen, L.busy, L.ewma, L.backlog);
    if (L.chg & CH_FRONT) rp[1] = make_int4(cap_l, en_l, L.fh, L.fn);
    if (lane == 0) {
      rp[2] = make_int4(L.P, next_id + nrows, t + 1, L.busy_mask);
    } else if (L.chg & CH_POOL) {
      recs[lane].P = L.P;
      recs[lane].busy_mask = L.busy_mask;
    }
    if (L.chg & CH_DONE) {
      if (RPM) rp[3] = make_int4(L.next_done, rpm_l, L.rcnt, inv_rpm_bits);
      else recs[lane].next_done = L.next_done;
    }
  }
  // Snapshot row for the next tick's route step: lane i < 4M writes
  // statistic i / M of model i % M, lanes m < M the validity bytes.
  if (ballot(ml && (L.chg & CH_STATS)) != 0) {
    float* row = a.snap + (size_t)e * snap_stride(M);
    const float inv_rpm_l = __int_as_float(inv_rpm_bits);
    // i / M for i < 4 M <= 128 as a multiply-high by ceil(2^32 / M)
    const uint32_t mmag = M == 1 ? 0u : 0xffffffffu / (uint32_t)M + 1u;
    for (int i0 = 0; i0 < 4 * M; i0 += 64) {
      const int i = i0 + lane;
      const int sidx = M == 1 ? i : (int)__umulhi((uint32_t)i, mmag), mm = i - sidx * M;
      const int srcm = mm < M ? mm : 0;
      const int32_t vq = shfl(L.qlen, srcm), vb = shfl(L.busy, srcm), vw = shfl(L.ewma, srcm),
                    vk = shfl(L.backlog, srcm);
      const float ib = __int_as_float(shfl(__float_as_int(inv_busy_l), srcm));
      const float ik = __int_as_float(shfl(__float_as_int(inv_back_l), srcm));
      const float v0 = RPM ? queue_stat(a, vq, shfl(rpm_l, srcm), shfl(L.rcnt, srcm),
                                        __int_as_float(shfl(__float_as_int(inv_rpm_l), srcm)))
                           : (float)vq * a.inv_qcap;
      const float v = sidx == 0 ? v0 : (sidx == 1 ? (float)vb * ib : (sidx == 2 ? (float)vw * a.inv_lat : (float)vk * ik));
      if (i < 4 * M) row[i] = v;
    }
    if (ml) {
      uint8_t* vb8 = (uint8_t*)(row + snap_valid_offset(M));
      vb8[lane] = (en_l != 0 && cap_l > 0 && L.qlen < a.qcap) ? 1 : 0;
    }
  }
  int64_t* envc_p = a.env_cnt + (size_t)e * kEnvCnt;
  if (nrows > 0) {
    int64_t* hist_p = a.hist + (size_t)e * a.A;
    if (lane < 2) counter_add(envc_p + lane, lane == 0 ? nrows : nomodel);
    if (lane < a.A) {
      const int32_t h = hist_s[lane];
      if (h != 0) counter_add(hist_p + lane, h);
    }
  }
  if constexpr (CHAIN) {
    if (lane == 0) a.pcnt[(size_t)((t + 1) & 1) * a.E + e] = pn;
    if (lane == 0 && q_done != 0) counter_add(envc_p + E_Q_DONE, q_done);
    if (lane == 0 && q_met != 0) counter_add(envc_p + E_Q_MET, q_met);
  }
}

// Dual update, step 1: exact int64 sums of completions and Q16 cost over every
// (env, model) counter row (order-independent: integer atomics).
// Chain pools count completed queries (env_cnt) instead of completed calls.
// Dual update (Sec. 4.4, Eq. 7) in one launch: every block sums its share of
// the completion and Q16 cost counters (waves by shuffles, the block through
// LDS) and adds them to acc[0..1] with one atomic each; the block that takes
// the last ticket (acc[2]) then finishes: over the completions since the
// previous update, C_bar = cost / (2^16 n) and lambda <- clip(lambda +
// eta (C_bar - 1), 0, lambda_max) in correctly rounded fp64 steps (no
// completion leaves lambda unchanged), and it resets acc for the next call.
__global__ __launch_bounds__(256) void dual_update_kernel(const int64_t* cnt, int64_t n_em,
                                                          const int64_t* env_cnt, int64_t n_env,
                                                          unsigned long long* acc, int64_t* last, double eta,
                                                          double lambda_max, double* lambda) {
  __shared__ unsigned long long part[2][4];
  __shared__ bool finisher;
  uint64_t n = 0, c = 0;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_em;
       i += (int64_t)gridDim.x * blockDim.x) {
    if (!env_cnt) n += (uint64_t)cnt[i * C_NUM + C_COMPLETED];
    c += (uint64_t)cnt[i * C_NUM + C_COST_Q16];
  }
  if (env_cnt) {
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n_env;
         i += (int64_t)gridDim.x * blockDim.x)
      n += (uint64_t)env_cnt[i * kEnvCnt + E_Q_DONE];
  }
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    n += (uint64_t)shfl_xor((int64_t)n, m);
    c += (uint64_t)shfl_xor((int64_t)c, m);
  }
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    part[0][w] = n;
    part[1][w] = c;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    uint64_t bn = 0, bc = 0;
    for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
      bn += part[0][i];
      bc += part[1][i];
    }
    if (bn != 0) atomicAdd(acc, (unsigned long long)bn);
    if (bc != 0) atomicAdd(acc + 1, (unsigned long long)bc);
    __threadfence();   // this block's sums are visible before its ticket
    finisher = atomicAdd(acc + 2, 1ull) == (unsigned long long)gridDim.x - 1;
  }
  __syncthreads();
  if (!finisher || threadIdx.x != 0) return;
  __threadfence();
  const int64_t tn = (int64_t)atomicAdd(acc, 0ull), tc = (int64_t)atomicAdd(acc + 1, 0ull);
  acc[0] = 0;
  acc[1] = 0;
  acc[2] = 0;
  const int64_t dn = tn - last[0], dc = tc - last[1];
  last[0] = tn;
  last[1] = tc;
  if (dn <= 0) return;
  {
    // one rounding per operation, as written (no fused multiply-add)
#pragma clang fp contract(off)
    const double cbar = (double)dc / (65536.0 * (double)dn);
    double l = *lambda + eta * (cbar - 1.0);
    l = l < 0.0 ? 0.0 : (l > lambda_max ? lambda_max : l);
    *lambda = l;
  }
}

}  // namespace

hipError_t launch_dual_update(const int64_t* cnt, int64_t n_em, const int64_t* env_cnt, int64_t n_env,
                              unsigned long long* acc, int64_t* last, double eta, double lambda_max,
                              double* lambda, hipStream_t s) {
  const int64_t n = n_em > n_env ? n_em : n_env;
  const int64_t want = (n + 255) / 256;
  const unsigned blocks = (unsigned)(want < 1024 ? (want < 1 ? 1 : want) : 1024);
  hipLaunchKernelGGL(dual_update_kernel, dim3(blocks), dim3(256), 0, s, cnt, n_em, env_cnt, n_env, acc, last,
                     eta, lambda_max, lambda);
  return hipGetLastError();
}

hipError_t launch_snapshot(const SchedArgs& a, int e0, int ne, hipStream_t s) {
  const int64_t n = (int64_t)ne * a.M;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(snapshot_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a, e0, ne);
  return hipGetLastError();
}

// Single-call pools load the fronts of two merging models at a time (the
// 5-wave register budget holds both); chain pools merge one model at a time.
hipError_t launch_schedule(const SchedArgs& a, bool rpm, bool chain, int waves_per_block, hipStream_t s) {
  const int w = waves_per_block == 1 || waves_per_block == 2 ? waves_per_block : 4;
  const unsigned blocks = (unsigned)(((int64_t)a.E + w - 1) / w);
  const dim3 threads(64 * w);
  if (chain) {
    if (rpm) hipLaunchKernelGGL((schedule_kernel<true, true, 1>), dim3(blocks), threads, 0, s, a);
    else hipLaunchKernelGGL((schedule_kernel<false, true, 1>), dim3(blocks), threads, 0, s, a);
  } else {
    if (rpm) hipLaunchKernelGGL((schedule_kernel<true, false, 2>), dim3(blocks), threads, 0, s, a);
    else hipLaunchKernelGGL((schedule_kernel<false, false, 2>), dim3(blocks), threads, 0, s, a);
  }
  return hipGetLastError();
}

}  // namespace im
