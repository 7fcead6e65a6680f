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

// Makes this wave's earlier global stores visible to its later loads.
__device__ __forceinline__ void wave_mem_sync() { __threadfence_block(); }

struct Queue {       // wave-uniform view of one (env, model) record
  int32_t qlen, busy, ewma, backlog, cap, enabled, fh, fn, P, busy_mask, next_done;
};

// Merge `lim` newcomers into the front held in registers (`fe`, lane i <
// q.fn), all of them below the front's largest key or the pool empty. `seg`
// is the model's sorted segment of a staged chunk in LDS (entries (key, id,
// svc | budget << 16, model)); newcomers arrive at tick t. The front followed
// by the reversed newcomers is a bitonic sequence of 128; its half-cleaner
// leaves the 64 smallest in `lo` (bitonic, sorted by one merge network) and
// the rest in `hi`, whose real entries spill to the pool.
__device__ __forceinline__ void merge_front(Queue& q, int4& fe, const int4* seg, int lim,
                                            int32_t t, int4* pool) {
  const int lane = lane_id();
  const int r = 63 - lane;
  int64_t kb = kKeyMax;
  int32_t pb[2] = {0, 0};
  if (r < lim) {
    const int4 v = seg[r];
    kb = composite(v.x, v.y);
    pb[0] = t;
    pb[1] = v.z;
  }
  const int64_t ka = lane < q.fn ? composite(fe.x, fe.y) : kKeyMax;
  const bool sw = kb < ka;
  int64_t klo = sw ? kb : ka;
  const int64_t khi = sw ? ka : kb;
  int32_t plo[2] = {sw ? pb[0] : fe.z, sw ? pb[1] : fe.w};
  const int32_t phi0 = sw ? fe.z : pb[0], phi1 = sw ? fe.w : pb[1];
  bitonic_merge64<2>(klo, plo);
  const int total = q.fn + lim;
  const int keep = total < kFront ? total : kFront;
  const bool spill = khi != kKeyMax;
  const uint64_t sm = ballot(spill);
  if (spill) pool[q.P + prefix_count(sm)] = make_int4(comp_key(khi), comp_id(khi), phi0, phi1);
  q.P += total - keep;
  q.fh = 0;
  q.fn = keep;
  fe = lane < keep ? make_int4(comp_key(klo), comp_id(klo), plo[0], plo[1]) : make_int4(0, 0, 0, 0);
}

// Refill the (empty) front with the min(64, P) smallest pool entries; the new
// front is returned in `fe` (lane i: entry i), the front array is not written.
// `pk`/`pi` are this wave's LDS staging rows (64 keys, 64 pool indices), `kb`
// its LDS buffer for 4 chunks of pool keys.
__device__ void refill(Queue& q, int4& fe, int4* pool, int64_t* pk, int32_t* pi, int2* kb) {
  const int lane = lane_id();
  const int P = q.P;
  wave_mem_sync();   // this tick's pool appends are read below
  if (P <= kFront) {
    int4 e = make_int4(0, 0, 0, 0);
    int64_t ck = kKeyMax;
    if (lane < P) { e = pool[lane]; ck = composite(e.x, e.y); }
    int32_t pay[2] = {e.z, e.w};
    bitonic_sort64<2>(ck, pay);
    fe = lane < P ? make_int4(comp_key(ck), comp_id(ck), pay[0], pay[1]) : make_int4(0, 0, 0, 0);
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
  constexpr int G = 4;   // pool chunks whose loads are in flight together
  const int2* keys = reinterpret_cast<const int2*>(pool);   // (key, id) of entry i at keys[2 i]
  for (int c0 = kFront; c0 < P; c0 += G * kFront) {
    int2 kv[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const int i = c0 + g * kFront + lane;
      kv[g] = i < P ? keys[2 * i] : make_int2(0x7fffffff, -1);   // (max, max) pads
    }
#pragma unroll
    for (int g = 0; g < G; ++g) kb[g * kFront + lane] = kv[g];
#pragma unroll 1
    for (int g = 0; g < G; ++g) {
      const int2 v = kb[g * kFront + lane];
      const int64_t kc = composite(v.x, v.y);
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
        pi[pos] = c0 + g * kFront + lane;
      }
      np += popc64(cm);
    }
  }
  if (np > 0) flush();
  const int sel = idx[0];
  fe = pool[sel];
  // Compact the pool: selected entries below the new size are holes, filled
  // with the unselected entries of the last 64 positions (same count).
  const int Pn = P - kFront;
  const uint64_t tail_sel = wave_or(sel >= Pn ? (1ull << (sel - Pn)) : 0ull);
  const uint64_t fillers = ~tail_sel;
  const uint64_t holes = ballot(sel < Pn);
  int4 fill = make_int4(0, 0, 0, 0);
  if (sel < Pn) {
    const int f = nth_set_bit(fillers, prefix_count(holes));
    fill = pool[Pn + f];
  }
  wave_mem_sync();
  if (sel < Pn) pool[sel] = fill;
  q.fh = 0;
  q.fn = kFront;
  q.P = Pn;
}

// Snapshot row entry of model m of env e from its state (one fp32 product
// per load statistic; validity byte). `part` selects which value to write
// (0..3: the four statistics, 4: validity), so lanes can share the work.
__device__ __forceinline__ void write_snap_part(const SchedArgs& a, int e, int m, int part,
                                                int32_t qlen, int32_t busy, int32_t ewma,
                                                int32_t backlog, int32_t cap, int32_t enabled) {
  float* row = a.snap + (size_t)e * snap_stride(a.M);
  const int c = cap < 0 ? 0 : (cap > IM_MAX_SLOTS ? IM_MAX_SLOTS : cap);
  switch (part) {
    case 0: row[m] = (float)qlen * a.inv_qcap; break;
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
    write_snap_part(a, e, m, part, r.qlen, r.busy, r.ewma, r.backlog, r.cap, r.enabled);
}

__device__ __forceinline__ int32_t wave_sum32(int32_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += shfl_xor(v, m);
  return v;
}

constexpr int kStageChunks = 4;   // arrival chunks (of 64) staged in LDS per round

// One wave per env. The env's arrivals are validated once; then, 64 at a time,
// they are partitioned by model (ballot + mbcnt ranks in id order give the
// tail-drop admission) and sorted once by (model, key, id) with a 64-lane
// bitonic network, so each model's newcomers form one sorted segment (a
// segmented sort). The sorted chunks are staged in LDS; each model then
// merges its segments into its queue, serves its slots and writes back.
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(4, 8))) void schedule_kernel(SchedArgs a) {
  __shared__ int4 stage[4][kStageChunks * 64];
  __shared__ int32_t hist_lds[4][IM_MAX_ACTIONS];
  __shared__ int32_t svc_lds[4][IM_MAX_MODELS];
  __shared__ int32_t acc_lds[4][IM_MAX_MODELS];
  __shared__ int64_t pend_k[4][kFront];   // refill candidate staging
  __shared__ int32_t pend_i[4][kFront];
  __shared__ int2 pend_kb[4][4 * kFront];
  const int lane = threadIdx.x & 63;
  const int wv = threadIdx.x >> 6;
  const int e = (int)blockIdx.x * 4 + wv;
  if (e >= a.E) return;
  int4* st = stage[wv];
  int32_t* hist_s = hist_lds[wv];
  int32_t* svc_s = svc_lds[wv];
  int32_t* acc_s = acc_lds[wv];
  hist_s[lane] = 0;                     // IM_MAX_ACTIONS == 64 lanes
  if (lane < IM_MAX_MODELS) { svc_s[lane] = 0; acc_s[lane] = 0; }
  const int M = a.M, K = a.K;

  // ---- validate the env's input; an invalid env is skipped this tick ----
  const int32_t lo = a.offsets[e], hi = a.offsets[e + 1];
  int32_t bad = 0;
  if (lo < 0 || hi < lo || hi > a.n_total || hi - lo > a.max_arrivals) bad = IM_ERR_COUNT;
  int32_t ac0 = -1, bu0 = 0, sv0 = 0;   // first chunk stays in registers
  if (!bad) {
    for (int32_t base = lo; base < hi; base += 64) {
      const int32_t i = base + lane;
      int32_t b = 0;
      if (i < hi) {
        const int32_t qi = a.q_idx[i];
        const int32_t bu = a.budget[i];
        const int32_t sv = a.base_svc[i];
        const int32_t ac = a.actions[i];
        if (qi < 0 || (int64_t)qi >= a.Q) b |= IM_ERR_QIDX;
        if (bu < 1) b |= IM_ERR_BUDGET;
        if (sv < 1 || sv > IM_SVC_MAX) b |= IM_ERR_SVC;
        if (ac < -1 || ac >= a.A) b |= IM_ERR_ACTION;
        if (base == lo) { ac0 = ac; bu0 = bu; sv0 = sv; }
      }
      // wave-wide OR of the five error bits, one ballot each
      if (ballot(b & IM_ERR_QIDX)) bad |= IM_ERR_QIDX;
      if (ballot(b & IM_ERR_BUDGET)) bad |= IM_ERR_BUDGET;
      if (ballot(b & IM_ERR_SVC)) bad |= IM_ERR_SVC;
      if (ballot(b & IM_ERR_ACTION)) bad |= IM_ERR_ACTION;
    }
  }
  ModelRec* recs = a.ms + (size_t)e * M;
  // The tick and the next request id live in the env's first record in
  // device memory, so a captured sequence of ticks replays with the right time.
  const int32_t t = recs[0].t;
  if (bad) {
    // The env's state is untouched and time still advances: busy slots keep
    // their remaining service, so their completion ticks move one tick later.
    if (lane == 0) {
      atomicOr(a.err, bad);
      recs[0].t = t + 1;
    }
    for (int m = 0; m < M; ++m) {
      if (recs[m].busy_mask == 0) continue;
      int4* sl = a.slots + (size_t)(e * M + m) * a.S;
      if (lane < a.S) {
        int4 v = sl[lane];
        if (v.x >= 0) {
          v.z += 1;
          sl[lane] = v;
        }
      }
      if (lane == 0) recs[m].next_done += 1;
    }
    return;
  }

  const int32_t n = hi - lo;
  // lane m < M: room left in model m's queue at the snapshot
  const int32_t room_l = lane < M ? a.qcap - recs[lane].qlen : 0;
  const int32_t next_id = recs[0].next_id;
  int64_t* hist_p = a.hist + (size_t)e * a.A;
  int32_t prior_l = 0;      // lane m: requests routed to model m so far (id order)
  int32_t acc_l = 0;        // lane m: requests accepted by model m so far
  int32_t nomodel = 0;
  // lane m: model m's load statistics after the tick, its capacity and
  // enable flag (for the snapshot row written once at the end)
  int32_t st_q = 0, st_b = 0, st_w = 0, st_k = 0, st_c = 0, st_en = 0;
  if (lane < M) {
    st_q = recs[lane].qlen; st_b = recs[lane].busy; st_w = recs[lane].ewma; st_k = recs[lane].backlog;
    st_c = recs[lane].cap; st_en = recs[lane].enabled;
  }
  bool snap_dirty = false;
  const int n_chunks = (n + 63) / 64;
  const int rounds = n_chunks > 0 ? (n_chunks + kStageChunks - 1) / kStageChunks : 1;

  for (int r = 0; r < rounds; ++r) {
    const int c0 = r * kStageChunks;
    const int nch = n_chunks - c0 < kStageChunks ? n_chunks - c0 : kStageChunks;
    // ---- partition, admission and one sort per chunk ----
    for (int c = 0; c < nch; ++c) {
      const int32_t base = lo + (c0 + c) * 64;
      const int32_t i = base + lane;
      const bool in = i < hi;
      int32_t ac = ac0, bu = bu0, sv = sv0;
      if (c0 + c != 0) {
        ac = in ? a.actions[i] : -1;
        bu = in ? a.budget[i] : 0;
        sv = in ? a.base_svc[i] : 0;
      }
      const int32_t mdl = ac >= 0 ? ac / K : -1;
      nomodel += popc64(ballot(in && ac < 0));
      if (in && ac >= 0) atomicAdd(&hist_s[ac], 1);   // routed requests per action
      int32_t rank = 0;
      for (int m = 0; m < M; ++m) {
        const uint64_t bal = ballot(in && mdl == m);
        if (bal == 0) continue;
        const int32_t pm = __builtin_amdgcn_readlane(prior_l, m);
        if (mdl == m) rank = pm + prefix_count(bal);
        if (lane == m) prior_l += popc64(bal);
      }
      const int32_t room = shfl(room_l, mdl >= 0 ? mdl : 0);
      const bool acc = in && mdl >= 0 && rank < room;
      const int32_t d = ac - mdl * K;
      const int32_t svc = sv * (d + 1);
      if (acc) {                                     // admitted count and service time per model
        atomicAdd(&acc_s[mdl], 1);
        atomicAdd(&svc_s[mdl], svc);
      }
      const int32_t key = a.key_mode == IM_KEY_DEADLINE ? t + bu
                          : (a.key_mode == IM_KEY_FCFS ? t : t + bu - svc);
      // sort key: model (63 for rejected rows) | key biased to unsigned | lane
      int64_t sk = (int64_t)(((uint64_t)(acc ? mdl : 63) << 38) |
                             ((uint64_t)((uint32_t)key ^ 0x80000000u) << 6) | (uint64_t)lane);
      int32_t pay[1] = {(int32_t)((uint32_t)svc | ((uint32_t)bu << 16))};
      bitonic_sort64<1>(sk, pay);
      const int32_t skey = (int32_t)((uint32_t)((uint64_t)sk >> 6) ^ 0x80000000u);
      const int32_t sid = next_id + (base - lo) + (int32_t)(sk & 63);
      st[c * 64 + lane] = make_int4(skey, sid, pay[0], (int32_t)((uint64_t)sk >> 38));
    }
    const bool last = r == rounds - 1;

    // lane m: newcomers admitted by model m this round and their service time
    const int32_t acc_round_l = lane < IM_MAX_MODELS ? acc_s[lane] : 0;
    const int32_t svc_round_l = lane < IM_MAX_MODELS ? svc_s[lane] : 0;
    if (lane < IM_MAX_MODELS) { acc_s[lane] = 0; svc_s[lane] = 0; }   // LDS accesses of one wave stay in order

    // ---- per model: insert its sorted segments, serve, write back ----
    // A model with no newcomers, no free slot to fill and no completion due
    // this tick is settled from its record alone: nothing is loaded or written.
    for (int m = 0; m < M; ++m) {
      const int em = e * M + m;
      ModelRec* rec = recs + m;
      Queue q;
      q.qlen = rec->qlen; q.busy = rec->busy; q.ewma = rec->ewma; q.backlog = rec->backlog;
      q.cap = rec->cap; q.enabled = rec->enabled; q.fh = rec->fh; q.fn = rec->fn;
      q.P = rec->P; q.busy_mask = rec->busy_mask; q.next_done = rec->next_done;
      const Queue q0 = q;
      int4* front = a.front + (size_t)em * kFront;
      int4* pool = a.pool + (size_t)em * a.qcap;
      const int32_t k_tot = __builtin_amdgcn_readlane(acc_round_l, m);   // newcomers admitted this round
      const int32_t svc_in = __builtin_amdgcn_readlane(svc_round_l, m);
      // The front is read only when it is needed; the live window
      // [fh, fh + fn) is rotated to lanes [0, fn) with lane shuffles.
      bool have_front = false;
      int4 fe = make_int4(0, 0, 0, 0);
      int fe_base = 0;                       // fe lane i mirrors front[fe_base + i]
      auto get_front = [&]() {
        const int4 all = front[lane];
        const int src = (q.fh + lane) & 63;
        fe.x = shfl((int32_t)all.x, src);
        fe.y = shfl((int32_t)all.y, src);
        fe.z = shfl((int32_t)all.z, src);
        fe.w = shfl((int32_t)all.w, src);
        if (lane >= q.fn) fe = make_int4(0, 0, 0, 0);
        fe_base = q.fh;
        have_front = true;
      };
      bool dirty = false;   // the front in registers differs from the front array
      if (k_tot > 0) {
        get_front();
        for (int c = 0; c < nch; ++c) {
          const int4 en = st[c * 64 + lane];
          const bool mine = en.w == m;
          const int k = popc64(ballot(mine));
          if (k == 0) continue;
          const int seg_lo = popc64(ballot(en.w < m));
          const int o = lane - seg_lo;   // offset in the model's sorted segment
          // newcomers merged into the front: those below its largest key, or
          // all of them while the pool is empty (the front then holds the queue)
          int lim;
          if (q.P == 0) {
            lim = k;
          } else if (q.fn == 0) {
            lim = 0;
          } else {
            const int64_t fmax = readlane64(composite(fe.x, fe.y), q.fn - 1);
            lim = popc64(ballot(mine && composite(en.x, en.y) < fmax));
          }
          if (mine && o >= lim) pool[q.P + o - lim] = make_int4(en.x, en.y, t, en.z);
          q.P += k - lim;
          if (lim > 0) {
            merge_front(q, fe, st + c * 64 + seg_lo, lim, t, pool);
            fe_base = 0;
            dirty = true;
          }
        }
        q.qlen += k_tot;
        q.backlog += svc_in;
        if (lane == m) acc_l += k_tot;
      }
      if (!last) {
        if (k_tot > 0) {
          if (dirty && lane >= q.fh - fe_base && lane < q.fh - fe_base + q.fn)
            front[fe_base + lane] = fe;   // the live window [fh, fh + fn)
          if (lane == 0) {
            rec->qlen = q.qlen; rec->backlog = q.backlog;
            rec->fh = q.fh; rec->fn = q.fn; rec->P = q.P;
          }
        }
        if (m == M - 1) wave_mem_sync();   // the next round re-reads these records
        continue;
      }

      // ---- service: fill free slots below c_m from the queue head ----
      const int capc = q.cap < a.S ? q.cap : a.S;
      const uint32_t free_m = ~(uint32_t)q.busy_mask & ((1u << capc) - 1u);
      const bool pops = free_m != 0 && q.qlen > 0;
      const bool due = q.busy_mask != 0 && q.next_done <= t;
      int32_t started = 0, wait_add = 0, svc_out = 0;
      int32_t completed = 0, slo_add = 0, lat_add = 0;
      if (pops || due) {
        // slot: {id, t_arr, tick of completion, budget}; id -1 = empty
        int4 sl = lane < a.S ? a.slots[(size_t)em * a.S + lane] : make_int4(-1, 0, 0, 0);
        if (pops) {
          if (!have_front) get_front();
          uint64_t empty = (uint64_t)free_m;
          while (empty != 0 && q.qlen > 0) {
            if (q.fn == 0) {
              refill(q, fe, pool, pend_k[wv], pend_i[wv], pend_kb[wv]);
              fe_base = 0;
              dirty = true;
            }
            if (q.fn == 0) break;   // unreachable while qlen == fn + P holds; never spin
            const int need = popc64(empty);
            const int take = need < q.fn ? need : q.fn;
            const int rnk = prefix_count(empty);
            const bool mine_slot = ((empty >> lane) & 1ull) && rnk < take;
            int4 en;
            const int src = (q.fh - fe_base + rnk) & 63;
            en.x = shfl((int32_t)fe.x, src);
            en.y = shfl((int32_t)fe.y, src);
            en.z = shfl((int32_t)fe.z, src);
            en.w = shfl((int32_t)fe.w, src);
            const int32_t svc = en.w & 0xffff;
            if (mine_slot) sl = make_int4(en.y, en.z, t + svc - 1, (int32_t)((uint32_t)en.w >> 16));
            uint64_t popped = ballot(mine_slot);
            empty &= ~popped;
            while (popped) {                       // at most max_slots lanes
              const int sp = __builtin_ctzll(popped);
              popped &= popped - 1;
              wait_add += t - __builtin_amdgcn_readlane(en.z, sp);
              svc_out += __builtin_amdgcn_readlane(svc, sp);
            }
            q.fh += take;
            q.fn -= take;
            q.qlen -= take;
            started += take;
          }
          q.backlog -= svc_out;
        }
        // ---- one tick of service; completions in slot order ----
        const bool busy_slot = lane < a.S && sl.x >= 0;
        const bool done = busy_slot && sl.z <= t;   // == t in every valid state
        const uint64_t done_mask = ballot(done);
        const int32_t lat = t - sl.y + 1;
        uint64_t dm = done_mask;
        int32_t ewma = q.ewma;
        while (dm) {
          const int s = __builtin_ctzll(dm);
          dm &= dm - 1;
          const int32_t ls = __builtin_amdgcn_readlane(lat, s);
          lat_add += ls;
          const int64_t delta = (int64_t)ls * 256 - ewma;
          const int64_t stepv = delta >= 0 ? (delta >> 3) : -((-delta + 7) >> 3);
          ewma = (int32_t)(ewma + stepv);
        }
        completed = popc64(done_mask);
        slo_add = popc64(ballot(done && lat <= sl.w));
        if (done) sl = make_int4(-1, 0, 0, 0);
        const uint64_t bm = ballot(lane < a.S && sl.x >= 0);
        q.busy = popc64(bm);
        q.busy_mask = (int32_t)(uint32_t)bm;
        q.ewma = ewma;
        // earliest completion tick among the busy slots (min over 8 lanes)
        int32_t nd = (lane < a.S && sl.x >= 0) ? sl.z : 0x7fffffff;
        nd = min(nd, xshfl<1>(nd));
        nd = min(nd, xshfl<2>(nd));
        nd = min(nd, xshfl<4>(nd));
        q.next_done = __builtin_amdgcn_readlane(nd, 0);
        if (lane < a.S) a.slots[(size_t)em * a.S + lane] = sl;
      }

      // ---- write back what changed ----
      if (dirty && lane >= q.fh - fe_base && lane < q.fh - fe_base + q.fn)
        front[fe_base + lane] = fe;   // the live window [fh, fh + fn)
      const bool stats = q.qlen != q0.qlen || q.busy != q0.busy || q.ewma != q0.ewma ||
                         q.backlog != q0.backlog;
      if (lane == 0 && (stats || q.fh != q0.fh || q.fn != q0.fn || q.P != q0.P ||
                        q.busy_mask != q0.busy_mask || q.next_done != q0.next_done)) {
        rec->qlen = q.qlen; rec->busy = q.busy; rec->ewma = q.ewma; rec->backlog = q.backlog;
        rec->fh = q.fh; rec->fn = q.fn; rec->P = q.P;
        rec->busy_mask = q.busy_mask; rec->next_done = q.next_done;
      }
      const int32_t routed_m = __builtin_amdgcn_readlane(prior_l, m);
      const int32_t acc_m = __builtin_amdgcn_readlane(acc_l, m);
      if (routed_m != 0 || started != 0 || completed != 0) {
        int64_t* cnt = a.cnt + (size_t)em * C_NUM;
        if (lane < C_NUM - 1) {
          int64_t add = 0;
          switch (lane) {
            case C_REJ_OVERFLOW: add = routed_m - acc_m; break;
            case C_ENQUEUED: add = acc_m; break;
            case C_STARTED: add = started; break;
            case C_COMPLETED: add = completed; break;
            case C_SLO_MET: add = slo_add; break;
            case C_LAT_SUM: add = lat_add; break;
            default: add = wait_add; break;
          }
          if (add != 0) cnt[lane] += add;
        }
      }
      if (lane == m) { st_q = q.qlen; st_b = q.busy; st_w = q.ewma; st_k = q.backlog; }
      snap_dirty |= stats;
    }
  }
  // Snapshot row for the next tick's route step: lane i < 4M writes
  // statistic i / M of model i % M, lanes m < M the validity bytes.
  if (snap_dirty) {
    float* row = a.snap + (size_t)e * snap_stride(M);
    for (int i0 = 0; i0 < 4 * M; i0 += 64) {
      const int i = i0 + lane;
      const int sidx = i / M, mm = i - sidx * M;
      const int32_t vq = shfl(st_q, mm), vb = shfl(st_b, mm), vw = shfl(st_w, mm), vk = shfl(st_k, mm);
      const int32_t cm = shfl(st_c, mm);
      const int c = cm < 0 ? 0 : (cm > IM_MAX_SLOTS ? IM_MAX_SLOTS : cm);
      if (i < 4 * M) {
        float v;
        switch (sidx) {
          case 0: v = (float)vq * a.inv_qcap; break;
          case 1: v = (float)vb * a.inv_tab[c]; break;
          case 2: v = (float)vw * a.inv_lat; break;
          default: v = (float)vk * a.inv_tab[IM_MAX_SLOTS + 1 + c]; break;
        }
        row[i] = v;
      }
    }
    if (lane < M) {
      uint8_t* vb8 = (uint8_t*)(row + snap_valid_offset(M));
      vb8[lane] = (st_en != 0 && st_c > 0 && st_q < a.qcap) ? 1 : 0;
    }
  }
  if (lane == 0) {
    recs[0].t = t + 1;
    if (n > 0) {
      recs[0].next_id = next_id + n;
      a.env_cnt[(size_t)e * 2] += n;
      a.env_cnt[(size_t)e * 2 + 1] += nomodel;
    }
  }
  if (n > 0 && lane < a.A) {
    const int32_t h = hist_s[lane];
    if (h != 0) hist_p[lane] += h;
  }
}

}  // namespace

hipError_t launch_snapshot(const SchedArgs& a, int e0, int ne, hipStream_t s) {
  const int64_t n = (int64_t)ne * a.M;
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(snapshot_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, a, e0, ne);
  return hipGetLastError();
}

hipError_t launch_schedule(const SchedArgs& a, hipStream_t s) {
  const int64_t waves = (int64_t)a.E;
  const unsigned blocks = (unsigned)((waves + 3) / 4);
  hipLaunchKernelGGL(schedule_kernel, dim3(blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace im
