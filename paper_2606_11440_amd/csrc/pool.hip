// Host side of libinframind: the C ABI declared in inframind.h.
//
// Owns the device state of a pool, packs the policy weights into the MFMA
// fragment order the route kernels read, validates arguments and launches the
// route / schedule kernels on the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "im_internal.h"
#include "inframind.h"

using im::ModelRec;

struct im_pool {
  im_pool_desc d{};
  int A = 0, S = 0, hidden = 0, n_layers = 0, out_tiles = 0, k1 = 0;
  int64_t Q = 0;
  int device = 0;
  const void* emb = nullptr;
  void* W[3] = {nullptr, nullptr, nullptr};
  float* bias[3] = {nullptr, nullptr, nullptr};
  float* inv_tab = nullptr;
  float inv_qcap = 0, inv_lat = 0, inv_bud = 0;
  ModelRec* ms = nullptr;
  int64_t* cnt = nullptr;
  int64_t* env_cnt = nullptr;
  int64_t* hist = nullptr;
  int4* slots = nullptr;
  int4* front = nullptr;
  int4* qpool = nullptr;
  uint8_t* rpm_ring = nullptr;              // [E*M*kRpmRing] per-tick dispatches, tick % 60
  float* snap = nullptr;
  int32_t* err = nullptr;
  int32_t* act_buf = nullptr;
  int64_t act_cap = 0;
  void* W_res = nullptr;                    // dual-pathway executor: resource-layer fragments
  float* dual_p = nullptr;                  // dual-pathway executor: fp32 parameter block
  unsigned long long* dual_acc = nullptr;   // [3] completions, Q16 cost, block tickets (zero between calls)
  int64_t* dual_last = nullptr;             // [2] totals at the previous dual update
  // multi-step chains: pending calls [2][E * pend_cap] and their counts
  // [2][E] (by tick parity), chain words of front, pool and slot entries, the
  // tick's rows (offsets, count, per-row query row, budget, role)
  bool chains = false;
  int32_t pend_cap = 0;
  int64_t rows_cap = 0;
  int4* pend = nullptr;
  int32_t* pcnt = nullptr;
  int2* front_ext = nullptr;
  int2* pool_ext = nullptr;
  int2* slot_ext = nullptr;
  int32_t* roff = nullptr;
  int32_t* n_rows = nullptr;
  int32_t* rq = nullptr;
  int16_t* rb = nullptr;
  int16_t* rr = nullptr;
  int32_t t = 0;
  int32_t cu_count = 0;
  int32_t route_blocks = -1;   // grid of the persistent route kernels (-1: one block per CU; 0: none)
  int32_t sched_waves = 4;     // envs per block of the schedule kernel
  int32_t* scratch = nullptr;  // this device's static actions staging (im_tick_noalloc)
  bool rpm_active = false;   // some model was given a rate limit (the windows are tracked from then on)
  std::string last_error;
};

static im::SchedArgs sched_args(im_pool* p);

namespace {

// Actions staging of im_tick_noalloc (one int32 per row of a tick, written by
// the route step and read by the schedule step), for callers that cannot
// allocate. A file-scope device array: every GPU the library runs on holds
// its own copy until the process ends, and calls on one GPU share it (each
// call overwrites every row it reads, so nothing has to start at zero; calls
// that overlap on one GPU race). In host code `scratch` names a host-side
// stand-in: its device address on the current device comes from
// hipGetSymbolAddress, resolved once per device (scratch_on) and used from
// then on.
constexpr int64_t kScratchRows = int64_t(1) << 21;   // 8 MiB
static __device__ __align__(256) int32_t scratch[kScratchRows];
std::mutex g_scratch_mu;
std::vector<int32_t*> g_scratch_dev;   // per device ordinal; nullptr until resolved

// The address of `scratch` on device `dev`, which must be the current device.
hipError_t scratch_on(int dev, int32_t** out) {
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (dev < 0) return hipErrorInvalidDevice;
  if ((size_t)dev >= g_scratch_dev.size()) g_scratch_dev.resize((size_t)dev + 1, nullptr);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_dev[dev] = static_cast<int32_t*>(ptr);
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

std::string g_create_error = "no error";

im_status fail(im_pool* p, im_status s, const std::string& msg) {
  if (p) p->last_error = msg; else g_create_error = msg;
  return s;
}

im_status hip_fail(im_pool* p, hipError_t e, const char* what) {
  return fail(p, e == hipErrorOutOfMemory ? IM_ENOMEM : IM_EHIP,
              std::string(what) + ": " + hipGetErrorString(e));
}

#define IM_HIP(p, call)                                   \
  do {                                                    \
    hipError_t _e = (call);                               \
    if (_e != hipSuccess) return hip_fail((p), _e, #call); \
  } while (0)

// fp32 -> bf16 bits, round to nearest even (NaN kept quiet).
uint16_t to_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// Input feature read by k-slot (kb, lane group g, element j) of a K block.
// Layer 0 reads the feature vector in natural order; deeper layers read the
// previous layer's accumulator registers, whose feature order inside each
// 16-wide block is 8*(j/4) + 4*g + j%4.
int bf16_k(int layer, int kb, int g, int j) {
  return layer == 0 ? 16 * kb + 8 * g + j : 16 * kb + 8 * (j >> 2) + 4 * g + (j & 3);
}
// Feature read by K step i of lane group q (lane / 16) in the fp32 kernel's
// 16x16x4 MFMA order: layer 1 in natural order; later layers in the previous
// layer's accumulator order (tile i / 4, register i % 4: feature 16 (i / 4)
// + 4 q + i % 4).
int f32_k(int layer, int i, int q) {
  return layer == 0 ? 4 * i + q : 16 * (i >> 2) + 4 * q + (i & 3);
}

template <class T>
im_status upload(im_pool* p, T** dst, const std::vector<T>& src) {
  IM_HIP(p, hipMalloc((void**)dst, std::max<size_t>(src.size(), 1) * sizeof(T)));
  if (!src.empty()) IM_HIP(p, hipMemcpy(*dst, src.data(), src.size() * sizeof(T), hipMemcpyHostToDevice));
  return IM_OK;
}

template <class T>
im_status zalloc(im_pool* p, T** dst, size_t n) {
  IM_HIP(p, hipMalloc((void**)dst, std::max<size_t>(n, 1) * sizeof(T)));
  IM_HIP(p, hipMemset(*dst, 0, std::max<size_t>(n, 1) * sizeof(T)));
  return IM_OK;
}

__global__ void set_field_kernel(int32_t* ptr, int32_t v) { *ptr = v; }
__global__ void set_rpm_kernel(ModelRec* r, int32_t limit, float inv) {
  r->rpm_limit = limit;
  r->inv_rpm = inv;
}

// Ring byte of tick tau (the device keeps the dispatches of tick tau at tau % 60).
inline int rpm_slot(int64_t tau) { return (int)(((tau % im::kRpmWindow) + im::kRpmWindow) % im::kRpmWindow); }

im_status check_arrivals(im_pool* p, const im_arrivals* arr) {
  if (!arr) return fail(p, IM_EINVAL, "arrivals is NULL");
  if (arr->n_total < 0) return fail(p, IM_EINVAL, "n_total < 0");
  if (!arr->offsets) return fail(p, IM_EINVAL, "offsets is NULL");
  if (arr->n_total > 0 && (!arr->q_idx || !arr->budget || !arr->base_svc))
    return fail(p, IM_EINVAL, "arrival field pointer is NULL");
  if (arr->n_total > 0 && p->d.net == IM_NET_DUAL && !arr->role)
    return fail(p, IM_EINVAL, "role is NULL (required by a dual-pathway pool)");
  if (arr->n_total > 0 && p->chains && !arr->n_steps)
    return fail(p, IM_EINVAL, "n_steps is NULL (required by a chain pool)");
  if ((int64_t)arr->n_total > (int64_t)p->d.n_envs * p->d.max_arrivals_per_env_tick)
    return fail(p, IM_EINVAL, "n_total exceeds n_envs * max_arrivals_per_env_tick");
  return IM_OK;
}

void free_pool(im_pool* p) {
  for (int l = 0; l < 3; ++l) {
    if (p->W[l]) (void)hipFree(p->W[l]);
    if (p->bias[l]) (void)hipFree(p->bias[l]);
  }
  void* bufs[] = {p->inv_tab, p->ms, p->cnt, p->env_cnt, p->hist, p->slots,
                  p->front, p->qpool, p->snap, p->err, p->act_buf, p->dual_acc, p->dual_last,
                  p->rpm_ring, p->W_res, p->dual_p, p->pend, p->pcnt, p->front_ext,
                  p->pool_ext, p->slot_ext, p->roff, p->n_rows, p->rq, p->rb, p->rr};
  for (void* b : bufs) if (b) (void)hipFree(b);
  delete p;
}

// Checks shared by both pool constructors (everything but the policy).
im_status check_desc_common(const im_pool_desc& d, int64_t n_queries, const int32_t* capacity) {
  const int A = d.n_models * d.n_depths;
  if (d.n_envs < 1 || d.n_models < 1 || d.n_models > IM_MAX_MODELS || d.n_depths < 1 ||
      d.n_depths > IM_MAX_DEPTHS || A > IM_MAX_ACTIONS)
    return fail(nullptr, IM_EINVAL, "n_envs/n_models/n_depths out of range");
  if (d.queue_cap < 1 || d.queue_cap > IM_MAX_QCAP) return fail(nullptr, IM_EINVAL, "queue_cap out of range");
  if (d.max_slots < 1 || d.max_slots > IM_MAX_SLOTS) return fail(nullptr, IM_EINVAL, "max_slots out of range");
  if (d.embed_dim < 1) return fail(nullptr, IM_EINVAL, "embed_dim < 1");
  if (d.value_head != 0 && d.value_head != 1) return fail(nullptr, IM_EINVAL, "value_head must be 0 or 1");
  if (d.key_mode < IM_KEY_SLACK || d.key_mode > IM_KEY_FCFS) return fail(nullptr, IM_EINVAL, "bad key_mode");
  if (d.max_arrivals_per_env_tick < 1) return fail(nullptr, IM_EINVAL, "max_arrivals_per_env_tick < 1");
  if (d.budget_max < 1) return fail(nullptr, IM_EINVAL, "budget_max < 1");
  if (n_queries < 1 || n_queries > INT32_MAX) return fail(nullptr, IM_EINVAL, "n_queries out of range");
  if (d.max_steps < 0 || d.max_steps > IM_MAX_STEPS) return fail(nullptr, IM_EINVAL, "max_steps out of range");
  if (d.max_steps > 1 && n_queries > (1 << 24))
    return fail(nullptr, IM_EUNSUPPORTED, "chain pools take at most 2^24 query-embedding rows");
  if (d.max_steps > 1 && d.net == IM_NET_DUAL && d.n_roles > 32)
    return fail(nullptr, IM_EUNSUPPORTED, "chain pools of the dual-pathway executor take at most 32 roles");
  for (int64_t i = 0; i < (int64_t)d.n_envs * d.n_models; ++i)
    if (capacity[i] < 0 || capacity[i] > d.max_slots)
      return fail(nullptr, IM_EINVAL, "capacity outside [0, max_slots]");
  return IM_OK;
}

im_pool* new_pool(const im_pool_desc& d, int64_t n_queries, const void* emb) {
  im_pool* p = new im_pool();
  p->d = d;
  p->A = d.n_models * d.n_depths;
  p->S = d.max_slots;
  p->chains = d.max_steps > 1;
  p->pend_cap = d.n_models * d.max_slots;
  p->Q = n_queries;
  p->emb = emb;
  (void)hipGetDevice(&p->device);
  if (hipDeviceGetAttribute(&p->cu_count, hipDeviceAttributeMultiprocessorCount, p->device) !=
      hipSuccess)
    p->cu_count = 0;
  // the static actions staging of this device (im_tick_noalloc reports its absence)
  if (scratch_on(p->device, &p->scratch) != hipSuccess) p->scratch = nullptr;
  return p;
}

// Feature reciprocals (each rounded once from fp64 to fp32), the zero state
// and the initial snapshot rows.
im_status init_state(im_pool* p, const int32_t* capacity, hipStream_t s) {
  const im_pool_desc& d = p->d;
  im_status st = IM_OK;
  p->inv_qcap = (float)(1.0 / d.queue_cap);
  p->inv_lat = (float)(1.0 / (256.0 * d.budget_max));
  p->inv_bud = (float)(1.0 / d.budget_max);
  {
    std::vector<float> tab(2 * (IM_MAX_SLOTS + 1));
    for (int c = 0; c <= IM_MAX_SLOTS; ++c) {
      const int cc = std::max(c, 1);
      tab[c] = (float)(1.0 / cc);
      tab[IM_MAX_SLOTS + 1 + c] = (float)(1.0 / ((double)cc * d.budget_max));
    }
    st = upload(p, &p->inv_tab, tab);
  }
  const size_t EM = (size_t)d.n_envs * d.n_models;
  if (st == IM_OK) {
    std::vector<ModelRec> recs(EM);
    std::memset(recs.data(), 0, EM * sizeof(ModelRec));
    for (size_t i = 0; i < EM; ++i) {
      recs[i].cap = capacity[i];
      recs[i].enabled = 1;
      recs[i].next_done = INT32_MAX;
    }
    st = upload(p, &p->ms, recs);
  }
  if (st == IM_OK) st = zalloc(p, &p->cnt, EM * im::C_NUM);
  if (st == IM_OK) st = zalloc(p, &p->env_cnt, (size_t)d.n_envs * im::kEnvCnt);
  if (st == IM_OK) st = zalloc(p, &p->hist, (size_t)d.n_envs * p->A);
  if (st == IM_OK) {
    std::vector<int4> sl(EM * d.max_slots, make_int4(-1, 0, 0, 0));
    st = upload(p, &p->slots, sl);
  }
  if (st == IM_OK) st = zalloc(p, &p->front, EM * im::kFront);
  if (st == IM_OK) st = zalloc(p, &p->qpool, EM * (size_t)d.queue_cap);
  if (st == IM_OK) st = zalloc(p, &p->rpm_ring, EM * (size_t)im::kRpmRing);
  if (st == IM_OK) st = zalloc(p, &p->snap, (size_t)d.n_envs * im::snap_stride(d.n_models));
  if (st == IM_OK) st = zalloc(p, &p->err, 1);
  if (st == IM_OK) st = zalloc(p, &p->dual_acc, 3);
  if (st == IM_OK) st = zalloc(p, &p->dual_last, 2);
  if (st == IM_OK && p->chains) {
    const size_t E = (size_t)d.n_envs;
    p->rows_cap = (int64_t)E * (d.max_arrivals_per_env_tick + p->pend_cap);
    st = zalloc(p, &p->pend, 2 * E * p->pend_cap);
    if (st == IM_OK) st = zalloc(p, &p->pcnt, 2 * E);
    if (st == IM_OK) st = zalloc(p, &p->front_ext, EM * im::kFront);
    if (st == IM_OK) st = zalloc(p, &p->pool_ext, EM * (size_t)d.queue_cap);
    if (st == IM_OK) st = zalloc(p, &p->slot_ext, EM * d.max_slots);
    if (st == IM_OK) st = zalloc(p, &p->roff, E + 1);
    if (st == IM_OK) st = zalloc(p, &p->n_rows, 2);
    if (st == IM_OK) st = zalloc(p, &p->rq, (size_t)p->rows_cap);
    if (st == IM_OK) st = zalloc(p, &p->rb, (size_t)p->rows_cap);
    if (st == IM_OK) st = zalloc(p, &p->rr, (size_t)p->rows_cap);
  }
  if (st == IM_OK) {
    p->act_cap = (int64_t)d.n_envs * d.max_arrivals_per_env_tick + (p->chains ? (int64_t)d.n_envs * p->pend_cap : 0);
    st = zalloc(p, &p->act_buf, (size_t)p->act_cap);
  }
  if (st == IM_OK) {
    hipError_t e = hipDeviceSynchronize();
    if (e == hipSuccess) e = im::launch_snapshot(sched_args(p), 0, d.n_envs, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) st = hip_fail(p, e, "initial snapshot");
  }
  return st;
}

}  // namespace

extern "C" {

im_status im_pool_create(const im_pool_desc* desc, const float* const* W, const float* const* b,
                         const void* emb, int64_t n_queries, const int32_t* capacity,
                         const float* logit_bias, void* stream, im_pool** out) {
  if (!desc || !W || !b || !emb || !capacity || !out)
    return fail(nullptr, IM_EINVAL, "NULL argument to im_pool_create");
  const im_pool_desc& d = *desc;
  im_status st0 = check_desc_common(d, n_queries, capacity);
  if (st0 != IM_OK) return st0;
  if (d.net != IM_NET_MLP) return fail(nullptr, IM_EINVAL, "net must be IM_NET_MLP (dual: im_pool_create_dual)");
  const int A = d.n_models * d.n_depths;
  if (d.feat_dim > IM_MAX_FEAT || d.feat_dim < d.embed_dim + 4 * d.n_models + 1)
    return fail(nullptr, IM_EINVAL, "feat_dim must be in [embed_dim + 4M + 1, IM_MAX_FEAT]");
  if (d.n_layers != 2 && d.n_layers != 3) return fail(nullptr, IM_EINVAL, "n_layers must be 2 or 3");
  if (d.widths[d.n_layers - 1] != A + d.value_head)
    return fail(nullptr, IM_EINVAL, "last width must be M*K + value_head");
  if (d.n_layers == 3 && d.widths[0] != d.widths[1])
    return fail(nullptr, IM_EUNSUPPORTED, "hidden widths must be equal");
  if (d.dtype != IM_F32 && d.dtype != IM_BF16) return fail(nullptr, IM_EINVAL, "bad dtype");
  const int H = d.widths[0];
  // output tiles of the last layer: 32 rows (bf16 kernels) or 16 rows (fp32)
  const int out_tiles = d.dtype == IM_F32 ? (A + d.value_head + 15) / 16 : (A + d.value_head + 31) / 32;
  if (!im::route_supported(d.dtype, H, d.n_layers, out_tiles))
    return fail(nullptr, IM_EUNSUPPORTED, "no route kernel for this dtype / hidden width");

  im_pool* p = new_pool(d, n_queries, emb);
  p->hidden = H;
  p->n_layers = d.n_layers;
  p->out_tiles = out_tiles;
  hipStream_t s = (hipStream_t)stream;
  im_status st = IM_OK;

  // ---- pack weights and biases into fragment order ----
  int in = d.feat_dim;
  for (int l = 0; l < d.n_layers && st == IM_OK; ++l) {
    const int outw = d.widths[l];
    const int TO = (outw + 31) / 32;
    const float* Wl = W[l];
    if (!Wl || !b[l]) { st = fail(p, IM_EINVAL, "NULL weight or bias"); break; }
    if (d.dtype == IM_BF16) {
      const int KB = (in + 15) / 16;
      if (l == 0) p->k1 = KB;
      std::vector<uint16_t> pk((size_t)TO * KB * 64 * 8, 0);
      for (int To = 0; To < TO; ++To)
        for (int kb = 0; kb < KB; ++kb)
          for (int lane = 0; lane < 64; ++lane)
            for (int j = 0; j < 8; ++j) {
              const int o = 32 * To + (lane & 31);
              const int k = bf16_k(l, kb, lane >> 5, j);
              if (o < outw && k < in)
                pk[(((size_t)To * KB + kb) * 64 + lane) * 8 + j] = to_bf16(Wl[(size_t)o * in + k]);
            }
      st = upload(p, (uint16_t**)&p->W[l], pk);
    } else {
      // 16-row output tiles, K steps of 4 grouped by four: [To][group][lane][4]
      const int TO16 = (outw + 15) / 16;
      const int KS = (in + 3) / 4, KG = (KS + 3) / 4;
      if (l == 0) p->k1 = KS;
      std::vector<float> pk((size_t)TO16 * KG * 64 * 4, 0.f);
      for (int To = 0; To < TO16; ++To)
        for (int i = 0; i < KS; ++i)
          for (int lane = 0; lane < 64; ++lane) {
            const int o = 16 * To + (lane & 15);
            const int k = f32_k(l, i, lane >> 4);
            if (o < outw && k < in)
              pk[(((size_t)To * KG + (i >> 2)) * 64 + lane) * 4 + (i & 3)] = Wl[(size_t)o * in + k];
          }
      st = upload(p, (float**)&p->W[l], pk);
    }
    if (st != IM_OK) break;
    // Bias in accumulator-register order: bf16 [To][g][v] -> feature 32To + 8(v/4) + 4g + v%4;
    // fp32 [To][q][r] -> feature 16To + 4q + r.
    const bool f32 = d.dtype == IM_F32;
    std::vector<float> bp((size_t)TO * 2 * 16, 0.f);   // TO 32-row tiles = 2 TO 16-row tiles
    for (size_t i = 0; i < bp.size(); ++i) {
      const int v = (int)(i % 16), g = (int)(i / 16) % 2, To = (int)(i / 32);
      const int o = f32 ? (int)i : 32 * To + 8 * (v >> 2) + 4 * g + (v & 3);
      if (o >= outw) continue;
      float val = b[l][o];
      if (l == d.n_layers - 1 && logit_bias && o < A) val += logit_bias[o / d.n_depths];
      bp[i] = val;
    }
    st = upload(p, &p->bias[l], bp);
    in = outw;
  }
  if (st == IM_OK) st = init_state(p, capacity, s);
  if (st != IM_OK) {
    g_create_error = p->last_error;
    free_pool(p);
    return st;
  }
  *out = p;
  return IM_OK;
}

im_status im_pool_create_dual(const im_pool_desc* desc, const im_dual_net* net, const void* emb,
                              int64_t n_queries, const int32_t* capacity, const float* logit_bias,
                              void* stream, im_pool** out) {
  if (!desc || !net || !emb || !capacity || !out)
    return fail(nullptr, IM_EINVAL, "NULL argument to im_pool_create_dual");
  const im_pool_desc& d = *desc;
  im_status st0 = check_desc_common(d, n_queries, capacity);
  if (st0 != IM_OK) return st0;
  if (d.net != IM_NET_DUAL) return fail(nullptr, IM_EINVAL, "net must be IM_NET_DUAL");
  if (d.n_roles < 1 || d.n_roles > IM_MAX_ROLES) return fail(nullptr, IM_EINVAL, "n_roles out of range");
  const float* need[] = {net->W_sem, net->b_sem, net->ln_sem_gain, net->ln_sem_bias, net->W_bud,
                         net->b_bud, net->W_sys, net->b_sys, net->W_res, net->b_res, net->ln_res_gain,
                         net->ln_res_bias, net->W_merge, net->b_merge, net->W_act, net->b_act,
                         net->role_emb};
  for (const float* q : need)
    if (!q) return fail(nullptr, IM_EINVAL, "NULL parameter in im_dual_net");
  if (d.dtype != IM_BF16) return fail(nullptr, IM_EUNSUPPORTED, "the dual-pathway executor runs in bf16 only");
  const int A = d.n_models * d.n_depths;
  const int Ao = A + d.value_head;
  if (!im::dual_supported(d.embed_dim, Ao) || d.n_models > im::kDualMaxModels)
    return fail(nullptr, IM_EUNSUPPORTED,
                "dual-pathway executor: embed_dim must be 64, 128, 256 or 384, M <= 16 and M*K + value_head <= 32");

  im_pool* p = new_pool(d, n_queries, emb);
  p->d.feat_dim = d.embed_dim + 4 * d.n_models + 1;
  p->d.n_layers = 0;
  hipStream_t s = (hipStream_t)stream;
  im_status st = IM_OK;
  const int Ed = d.embed_dim, M = d.n_models, KBQ = Ed / 16;
  using im::kDualSem;
  using im::kDualRes;
  using im::kDualMerge;
  // query half of W_sem: K step kb = 4 G + i of lane half g holds elements
  // 64 G + 32 g + 8 i + j (each lane reads 64 contiguous bytes per group)
  {
    std::vector<uint16_t> pk((size_t)4 * KBQ * 64 * 8);
    for (int T = 0; T < 4; ++T)
      for (int kb = 0; kb < KBQ; ++kb)
        for (int lane = 0; lane < 64; ++lane)
          for (int j = 0; j < 8; ++j) {
            const int o = 32 * T + (lane & 31);
            const int k = 64 * (kb >> 2) + 32 * (lane >> 5) + 8 * (kb & 3) + j;
            pk[(((size_t)T * KBQ + kb) * 64 + lane) * 8 + j] = to_bf16(net->W_sem[(size_t)o * 2 * Ed + k]);
          }
    st = upload(p, (uint16_t**)&p->W[0], pk);
  }
  // fragments of a layer whose input is (layer > 0) a previous accumulator or
  // (layer == 0) a vector in natural order
  auto pack = [&](const float* Wm, int outw, int in, int layer, int TO, void** dst) {
    const int KB = in / 16;
    std::vector<uint16_t> pk((size_t)TO * KB * 64 * 8, 0);
    for (int T = 0; T < TO; ++T)
      for (int kb = 0; kb < KB; ++kb)
        for (int lane = 0; lane < 64; ++lane)
          for (int j = 0; j < 8; ++j) {
            const int o = 32 * T + (lane & 31);
            const int k = bf16_k(layer, kb, lane >> 5, j);
            if (o < outw) pk[(((size_t)T * KB + kb) * 64 + lane) * 8 + j] = to_bf16(Wm[(size_t)o * in + k]);
          }
    return upload(p, (uint16_t**)dst, pk);
  };
  if (st == IM_OK) st = pack(net->W_merge, kDualMerge, kDualSem + kDualRes, 1, 4, &p->W[1]);
  if (st == IM_OK) st = pack(net->W_act, Ao, kDualMerge, 1, 1, &p->W[2]);
  if (st == IM_OK) st = pack(net->W_res, kDualRes, 32, 0, 2, &p->W_res);
  // fp32 parameter block
  const int roff = im::DP_ROLE;
  std::vector<float> dp((size_t)roff + (size_t)d.n_roles * kDualSem, 0.f);
  auto acc_order = [&](int off, const float* v, int width, int tiles, bool logit) {
    for (int T = 0; T < tiles; ++T)
      for (int g = 0; g < 2; ++g)
        for (int vv = 0; vv < 16; ++vv) {
          const int o = 32 * T + 8 * (vv >> 2) + 4 * g + (vv & 3);
          if (o >= width) continue;
          float x = v[o];
          if (logit && logit_bias && o < A) x += logit_bias[o / d.n_depths];
          dp[off + (T * 2 + g) * 16 + vv] = x;
        }
  };
  auto bfv = [](float x) {
    const uint32_t u = (uint32_t)to_bf16(x) << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
  };
  acc_order(im::DP_LN_SEM_G, net->ln_sem_gain, kDualSem, 4, false);
  acc_order(im::DP_LN_SEM_B, net->ln_sem_bias, kDualSem, 4, false);
  acc_order(im::DP_B_RES, net->b_res, kDualRes, 2, false);
  acc_order(im::DP_LN_RES_G, net->ln_res_gain, kDualRes, 2, false);
  acc_order(im::DP_LN_RES_B, net->ln_res_bias, kDualRes, 2, false);
  acc_order(im::DP_B_MERGE, net->b_merge, kDualMerge, 4, false);
  acc_order(im::DP_B_ACT, net->b_act, Ao, 1, true);
  for (int k = 0; k < 16; ++k) {
    dp[im::DP_W_BUD + k] = bfv(net->W_bud[k]);
    dp[im::DP_B_BUD + k] = net->b_bud[k];
    dp[im::DP_B_SYS + k] = net->b_sys[k];
  }
  // system head column of snapshot feature k = stat * M + m: the paper's
  // input order is [queue depth | end-to-end latency | KV-cache use], the
  // snapshot's [queue depth | busy / c_m | latency EWMA]
  for (int k = 0; k < 3 * M; ++k) {
    const int stat = k / M, m = k % M;
    const int col = stat == 0 ? m : (stat == 1 ? 2 * M + m : M + m);
    for (int r = 0; r < 16; ++r) dp[im::DP_W_SYS + k * 16 + r] = bfv(net->W_sys[(size_t)r * 3 * M + col]);
  }
  if (st == IM_OK) st = upload(p, &p->dual_p, dp);
  // role projections b_sem + W_sem[:, E_d:] e_r, computed on the device
  if (st == IM_OK) {
    std::vector<uint16_t> wr((size_t)kDualSem * Ed), rt((size_t)d.n_roles * Ed);
    for (int o = 0; o < kDualSem; ++o)
      for (int k = 0; k < Ed; ++k) wr[(size_t)o * Ed + k] = to_bf16(net->W_sem[(size_t)o * 2 * Ed + Ed + k]);
    for (size_t i = 0; i < rt.size(); ++i) rt[i] = to_bf16(net->role_emb[i]);
    uint16_t *dwr = nullptr, *drt = nullptr;
    float* dbs = nullptr;
    std::vector<float> bs(net->b_sem, net->b_sem + kDualSem);
    st = upload(p, &dwr, wr);
    if (st == IM_OK) st = upload(p, &drt, rt);
    if (st == IM_OK) st = upload(p, &dbs, bs);
    if (st == IM_OK) {
      hipError_t e = im::launch_role_projection(dwr, drt, dbs, d.n_roles, Ed, p->dual_p + roff, s);
      if (e == hipSuccess) e = hipStreamSynchronize(s);
      if (e != hipSuccess) st = hip_fail(p, e, "role projection");
    }
    if (dwr) (void)hipFree(dwr);
    if (drt) (void)hipFree(drt);
    if (dbs) (void)hipFree(dbs);
  }
  if (st == IM_OK) st = init_state(p, capacity, s);
  if (st != IM_OK) {
    g_create_error = p->last_error;
    free_pool(p);
    return st;
  }
  *out = p;
  return IM_OK;
}

void im_destroy(im_pool* p) {
  if (!p) return;
  (void)hipDeviceSynchronize();
  free_pool(p);
}

static im::RouteArgs route_args(im_pool* p, const im_arrivals* arr, int32_t* actions, float* logits) {
  im::RouteArgs a{};
  a.offsets = arr->offsets;
  a.q_idx = arr->q_idx;
  a.budget = arr->budget;
  a.n_total = arr->n_total;
  a.E = p->d.n_envs;
  a.M = p->d.n_models;
  a.K = p->d.n_depths;
  a.A = p->A;
  a.embed_dim = p->d.embed_dim;
  a.feat_dim = p->d.feat_dim;
  a.k1 = p->k1;
  a.qcap = p->d.queue_cap;
  a.Q = p->Q;
  a.emb = p->emb;
  for (int l = 0; l < 3; ++l) { a.W[l] = p->W[l]; a.bias[l] = p->bias[l]; }
  a.ms = p->ms;
  a.snap = p->snap;
  a.inv_bud = p->inv_bud;
  a.actions = actions;
  a.logits = logits;
  a.err = p->err;
  a.persistent_blocks = p->route_blocks < 0 ? p->cu_count : p->route_blocks;
  a.net = p->d.net;
  if (p->d.net == IM_NET_DUAL) {
    a.role = arr->role;
    a.n_roles = p->d.n_roles;
    a.W_res = p->W_res;
    a.dual_p = p->dual_p;
  }
  if (p->chains) {
    // the tick's rows (pending calls, then arrivals) built on the device;
    // their count is read there, n_total bounds it
    a.offsets = p->roff;
    a.q_idx = p->rq;
    a.budget = p->rb;
    a.role = p->d.net == IM_NET_DUAL ? p->rr : nullptr;
    a.n_total = arr->n_total + p->d.n_envs * p->pend_cap;
    a.n_total_dev = p->n_rows;
  }
  a.envs_per_row = a.n_total > 0 ? (float)((double)p->d.n_envs / a.n_total) : 0.f;
  return a;
}

// Chain pools: the tick's rows from the pending calls and the arrivals.
static hipError_t build_rows(im_pool* p, const im_arrivals* arr, hipStream_t s) {
  im::RowsArgs r{};
  r.offsets = arr->offsets;
  r.n_total = arr->n_total;
  r.E = p->d.n_envs;
  r.M = p->d.n_models;
  r.max_arrivals = p->d.max_arrivals_per_env_tick;
  r.pend_cap = p->pend_cap;
  r.n_roles = p->d.net == IM_NET_DUAL ? p->d.n_roles : 0;
  r.q_idx = arr->q_idx;
  r.budget = arr->budget;
  r.role = p->d.net == IM_NET_DUAL ? arr->role : nullptr;
  r.ms = p->ms;
  r.pend = p->pend;
  r.pcnt = p->pcnt;
  r.roff = p->roff;
  r.n_rows = p->n_rows;
  r.rq = p->rq;
  r.rb = p->rb;
  r.rr = p->rr;
  return im::launch_rows(r, s);
}

static im_status route_impl(im_pool* p, const im_arrivals* arr, im::RouteArgs a, hipStream_t s) {
  if (p->chains) IM_HIP(p, build_rows(p, arr, s));
  IM_HIP(p, im::launch_route(a, p->d.dtype, p->hidden, p->n_layers, p->out_tiles, s));
  return IM_OK;
}

im_status im_route(im_pool* p, const im_arrivals* arr, int32_t* actions, float* logits,
                   void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  im_status st = check_arrivals(p, arr);
  if (st != IM_OK) return st;
  if ((arr->n_total > 0 || p->chains) && !actions) return fail(p, IM_EINVAL, "actions is NULL");
  return route_impl(p, arr, route_args(p, arr, actions, logits), (hipStream_t)stream);
}

im_status im_route_sample(im_pool* p, const im_arrivals* arr, uint64_t seed, int32_t greedy,
                          const im_policy_out* out, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  im_status st = check_arrivals(p, arr);
  if (st != IM_OK) return st;
  if (!out) return fail(p, IM_EINVAL, "out is NULL");
  if ((arr->n_total > 0 || p->chains) && !out->actions) return fail(p, IM_EINVAL, "actions is NULL");
  if (out->value && !p->d.value_head) return fail(p, IM_EINVAL, "value requested from a pool without a value head");
  im::RouteArgs a = route_args(p, arr, out->actions, out->logits);
  a.rl = 1;
  a.greedy = greedy ? 1 : 0;
  a.seed_lo = (uint32_t)seed;
  a.seed_hi = (uint32_t)(seed >> 32);
  a.logp = out->logp;
  a.entropy = out->entropy;
  a.value = out->value;
  return route_impl(p, arr, a, (hipStream_t)stream);
}

// build: rebuild the chain pool's rows first (not needed right after a route
// of the same tick).
static im_status schedule_impl(im_pool* p, const im_arrivals* arr, const int32_t* actions, bool build,
                               hipStream_t s) {
  if (p->t == INT32_MAX - 65536) return fail(p, IM_EINVAL, "tick counter exhausted");
  im::SchedArgs a = sched_args(p);
  a.offsets = arr->offsets;
  a.q_idx = arr->q_idx;
  a.budget = arr->budget;
  a.base_svc = arr->base_svc;
  a.actions = actions;
  a.n_total = arr->n_total;
  if (p->d.net == IM_NET_DUAL) {
    a.role = arr->role;
    a.n_roles = p->d.n_roles;
  }
  if (p->chains) {
    if (build) IM_HIP(p, build_rows(p, arr, s));
    a.n_steps = arr->n_steps;
    a.max_steps = p->d.max_steps;
    a.pend_cap = p->pend_cap;
    a.roff = p->roff;
    a.pend = p->pend;
    a.pcnt = p->pcnt;
    a.front_ext = p->front_ext;
    a.pool_ext = p->pool_ext;
    a.slot_ext = p->slot_ext;
    a.csr_bad = p->n_rows + 1;
  }
  IM_HIP(p, im::launch_schedule(a, p->rpm_active, p->chains, p->sched_waves, s));
  p->t += 1;
  return IM_OK;
}

im_status im_schedule(im_pool* p, const im_arrivals* arr, const int32_t* actions, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  im_status st = check_arrivals(p, arr);
  if (st != IM_OK) return st;
  if ((arr->n_total > 0 || p->chains) && !actions) return fail(p, IM_EINVAL, "actions is NULL");
  return schedule_impl(p, arr, actions, true, (hipStream_t)stream);
}

static im::SchedArgs sched_args(im_pool* p) {
  im::SchedArgs a{};
  a.E = p->d.n_envs;
  a.M = p->d.n_models;
  a.K = p->d.n_depths;
  a.A = p->A;
  a.S = p->S;
  a.qcap = p->d.queue_cap;
  a.max_arrivals = p->d.max_arrivals_per_env_tick;
  a.key_mode = p->d.key_mode;
  a.Q = p->Q;
  a.ms = p->ms;
  a.cnt = p->cnt;
  a.env_cnt = p->env_cnt;
  a.hist = p->hist;
  a.slots = p->slots;
  a.front = p->front;
  a.pool = p->qpool;
  a.rpm_ring = p->rpm_ring;
  a.err = p->err;
  a.snap = p->snap;
  a.inv_qcap = p->inv_qcap;
  a.inv_lat = p->inv_lat;
  a.inv_tab = p->inv_tab;
  return a;
}

im_status im_tick(im_pool* p, const im_arrivals* arr, int32_t* actions_out, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  im_status st = check_arrivals(p, arr);
  if (st != IM_OK) return st;
  int32_t* act = actions_out ? actions_out : p->act_buf;
  st = route_impl(p, arr, route_args(p, arr, act, nullptr), (hipStream_t)stream);
  if (st != IM_OK) return st;
  return schedule_impl(p, arr, act, false, (hipStream_t)stream);
}

im_status im_tick_noalloc(im_pool* p, const im_arrivals* arr, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  im_status st = check_arrivals(p, arr);
  if (st != IM_OK) return st;
  // rows of the tick: the arrivals, and a chain pool's pending calls on top
  const int64_t rows = (int64_t)arr->n_total + (p->chains ? (int64_t)p->d.n_envs * p->pend_cap : 0);
  if (rows > kScratchRows)
    return fail(p, IM_EINVAL, "im_tick_noalloc: the tick's rows (" + std::to_string(rows) +
                                  ") exceed its static staging of 2^21 rows; use im_tick");
  if (!p->scratch) return fail(p, IM_EHIP, "im_tick_noalloc: static staging unavailable on this device");
  int32_t* act = p->scratch;
  st = route_impl(p, arr, route_args(p, arr, act, nullptr), (hipStream_t)stream);
  if (st != IM_OK) return st;
  return schedule_impl(p, arr, act, false, (hipStream_t)stream);
}

im_status im_get_rows(im_pool* p, im_rows* out) {
  if (!p || !out) return fail(p, IM_EINVAL, "NULL argument to im_get_rows");
  if (!p->chains) return fail(p, IM_EINVAL, "im_get_rows: not a chain pool");
  out->offsets = p->roff;
  out->n_rows = p->n_rows;
  out->q_idx = p->rq;
  out->budget = p->rb;
  out->role = p->rr;
  return IM_OK;
}

im_status im_dual_update(im_pool* p, double eta, double lambda_max, double* lambda, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (!lambda) return fail(p, IM_EINVAL, "lambda is NULL");
  if (!(eta >= 0.0) || !(lambda_max >= 0.0)) return fail(p, IM_EINVAL, "eta and lambda_max must be >= 0");
  IM_HIP(p, im::launch_dual_update(p->cnt, (int64_t)p->d.n_envs * p->d.n_models,
                                   p->chains ? p->env_cnt : nullptr, p->d.n_envs, p->dual_acc,
                                   p->dual_last, eta, lambda_max, lambda, (hipStream_t)stream));
  return IM_OK;
}

im_status im_set_enabled(im_pool* p, int32_t env, int32_t model, int32_t enabled, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (env < 0 || env >= p->d.n_envs || model < 0 || model >= p->d.n_models)
    return fail(p, IM_EINVAL, "env/model out of range");
  ModelRec* r = p->ms + (size_t)env * p->d.n_models + model;
  hipLaunchKernelGGL(set_field_kernel, dim3(1), dim3(1), 0, (hipStream_t)stream, &r->enabled,
                     enabled ? 1 : 0);
  IM_HIP(p, hipGetLastError());
  IM_HIP(p, im::launch_snapshot(sched_args(p), env, 1, (hipStream_t)stream));
  return IM_OK;
}

im_status im_set_capacity(im_pool* p, int32_t env, int32_t model, int32_t capacity, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (env < 0 || env >= p->d.n_envs || model < 0 || model >= p->d.n_models)
    return fail(p, IM_EINVAL, "env/model out of range");
  if (capacity < 0 || capacity > p->S) return fail(p, IM_EINVAL, "capacity outside [0, max_slots]");
  ModelRec* r = p->ms + (size_t)env * p->d.n_models + model;
  hipLaunchKernelGGL(set_field_kernel, dim3(1), dim3(1), 0, (hipStream_t)stream, &r->cap, capacity);
  IM_HIP(p, hipGetLastError());
  IM_HIP(p, im::launch_snapshot(sched_args(p), env, 1, (hipStream_t)stream));
  return IM_OK;
}

im_status im_set_rpm_limit(im_pool* p, int32_t env, int32_t model, int32_t rpm_limit, void* stream) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (env < 0 || env >= p->d.n_envs || model < 0 || model >= p->d.n_models)
    return fail(p, IM_EINVAL, "env/model out of range");
  if (rpm_limit < 0 || rpm_limit > (1 << 30)) return fail(p, IM_EINVAL, "rpm_limit outside [0, 2^30]");
  ModelRec* r = p->ms + (size_t)env * p->d.n_models + model;
  const float inv = rpm_limit > 0 ? (float)(1.0 / rpm_limit) : 0.f;   // rounded once from fp64
  if (rpm_limit > 0) p->rpm_active = true;
  hipLaunchKernelGGL(set_rpm_kernel, dim3(1), dim3(1), 0, (hipStream_t)stream, r, rpm_limit, inv);
  IM_HIP(p, hipGetLastError());
  IM_HIP(p, im::launch_snapshot(sched_args(p), env, 1, (hipStream_t)stream));
  return IM_OK;
}

im_status im_set_launch(im_pool* p, int32_t route_blocks, int32_t sched_waves) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (route_blocks < -1) return fail(p, IM_EINVAL, "route_blocks < -1");
  if (sched_waves != 0 && sched_waves != 1 && sched_waves != 2 && sched_waves != 4)
    return fail(p, IM_EINVAL, "sched_waves not in {0, 1, 2, 4}");
  p->route_blocks = route_blocks;
  if (sched_waves) p->sched_waves = sched_waves;
  return IM_OK;
}

im_status im_get_error(im_pool* p, int32_t* bits) {
  if (!p || !bits) return fail(p, IM_EINVAL, "NULL argument");
  IM_HIP(p, hipDeviceSynchronize());
  IM_HIP(p, hipMemcpy(bits, p->err, sizeof(int32_t), hipMemcpyDeviceToHost));
  return *bits ? IM_EDEVICE : IM_OK;
}

im_status im_clear_error(im_pool* p) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  IM_HIP(p, hipDeviceSynchronize());
  IM_HIP(p, hipMemset(p->err, 0, sizeof(int32_t)));
  IM_HIP(p, hipDeviceSynchronize());
  return IM_OK;
}

const char* im_last_error(const im_pool* p) {
  return p ? p->last_error.c_str() : g_create_error.c_str();
}

im_status im_read_state(im_pool* p, int32_t env_begin, int32_t env_count, int32_t* tick,
                        im_env_state* envs, im_model_state* models, im_slot* slots,
                        im_entry* queues, int64_t* hist) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (env_begin < 0 || env_count < 0 || (int64_t)env_begin + env_count > p->d.n_envs)
    return fail(p, IM_EINVAL, "env range out of bounds");
  IM_HIP(p, hipDeviceSynchronize());
  const int M = p->d.n_models, S = p->S, qcap = p->d.queue_cap, A = p->A;
  const size_t em0 = (size_t)env_begin * M, EMc = (size_t)env_count * M;
  std::vector<ModelRec> recs(EMc);
  std::vector<int64_t> cnt(EMc * im::C_NUM);
  if (EMc) {
    IM_HIP(p, hipMemcpy(recs.data(), p->ms + em0, EMc * sizeof(ModelRec), hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(cnt.data(), p->cnt + em0 * im::C_NUM, cnt.size() * 8, hipMemcpyDeviceToHost));
    p->t = recs[0].t;   // every env advances every tick; graph replays advance it too
  }
  if (tick) *tick = p->t;
  if (envs && env_count) {
    constexpr int EC = im::kEnvCnt;
    std::vector<int64_t> ec((size_t)env_count * EC);
    IM_HIP(p, hipMemcpy(ec.data(), p->env_cnt + (size_t)env_begin * EC, ec.size() * 8,
                        hipMemcpyDeviceToHost));
    for (int e = 0; e < env_count; ++e) {
      envs[e].arrived = ec[EC * e + im::E_ARRIVED];
      envs[e].rej_nomodel = ec[EC * e + im::E_REJ_NOMODEL];
      envs[e].next_id = recs[(size_t)e * M].next_id;
      envs[e]._pad = 0;
      envs[e].q_done = ec[EC * e + im::E_Q_DONE];
      envs[e].q_met = ec[EC * e + im::E_Q_MET];
    }
  }
  if (models) {
    for (size_t i = 0; i < EMc; ++i) {
      im_model_state& o = models[i];
      std::memset(&o, 0, sizeof(o));
      o.qlen = recs[i].qlen; o.busy = recs[i].busy; o.ewma_q8 = recs[i].ewma;
      o.backlog = recs[i].backlog; o.capacity = recs[i].cap; o.enabled = recs[i].enabled;
      const int64_t* c = &cnt[i * im::C_NUM];
      o.rej_overflow = c[im::C_REJ_OVERFLOW]; o.enqueued = c[im::C_ENQUEUED];
      o.started = c[im::C_STARTED]; o.completed = c[im::C_COMPLETED]; o.slo_met = c[im::C_SLO_MET];
      o.lat_sum = c[im::C_LAT_SUM]; o.wait_sum = c[im::C_WAIT_SUM];
      o.cost_q16 = c[im::C_COST_Q16];
      o.rpm_limit = recs[i].rpm_limit;
      o.rpm_count = recs[i].rpm_count;
    }
    std::vector<uint8_t> ring(EMc * im::kRpmRing);
    if (EMc)
      IM_HIP(p, hipMemcpy(ring.data(), p->rpm_ring + em0 * im::kRpmRing, ring.size(), hipMemcpyDeviceToHost));
    for (size_t i = 0; i < EMc; ++i)
      for (int k = 0; k < im::kRpmWindow; ++k)
        models[i].rpm_hist[k] = (int64_t)p->t - 1 - k >= 0 ? ring[i * im::kRpmRing + rpm_slot((int64_t)p->t - 1 - k)] : 0;
  }
  if (slots && EMc) {
    // The device keeps a busy slot's completion tick; the state reports the
    // service ticks left after the env's last completed tick.
    std::vector<int4> sl(EMc * S);
    IM_HIP(p, hipMemcpy(sl.data(), p->slots + em0 * S, sl.size() * sizeof(int4), hipMemcpyDeviceToHost));
    for (size_t i = 0; i < EMc; ++i) {
      const int32_t t_env = recs[(i / M) * M].t;
      for (int s = 0; s < S; ++s) {
        const int4 v = sl[i * S + s];
        im_slot& o = slots[i * S + s];
        if (v.x >= 0) { o.id = v.x; o.t_arr = v.y; o.rem = v.z - t_env + 1; o.budget = v.w; }
        else { o.id = -1; o.t_arr = 0; o.rem = 0; o.budget = 0; }
      }
    }
  }
  if (hist && env_count)
    IM_HIP(p, hipMemcpy(hist, p->hist + (size_t)env_begin * A, (size_t)env_count * A * 8,
                        hipMemcpyDeviceToHost));
  if (queues && EMc) {
    // Materialise each queue in service order: the sorted front, then the
    // pool sorted by (key, id) (every pool key exceeds every front key).
    std::vector<int4> fr(EMc * im::kFront), pl(EMc * (size_t)qcap);
    IM_HIP(p, hipMemcpy(fr.data(), p->front + em0 * im::kFront, fr.size() * sizeof(int4),
                        hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(pl.data(), p->qpool + em0 * qcap, pl.size() * sizeof(int4),
                        hipMemcpyDeviceToHost));
    std::memset(queues, 0, EMc * qcap * sizeof(im_entry));
    std::vector<int4> tmp;
    for (size_t i = 0; i < EMc; ++i) {
      const ModelRec& r = recs[i];
      tmp.assign(fr.begin() + i * im::kFront + r.fh, fr.begin() + i * im::kFront + r.fh + r.fn);
      const size_t f = tmp.size();
      tmp.insert(tmp.end(), pl.begin() + i * qcap, pl.begin() + i * qcap + r.P);
      std::sort(tmp.begin() + f, tmp.end(), [](const int4& x, const int4& y) {
        return x.x != y.x ? x.x < y.x : x.y < y.y;
      });
      im_entry* q = queues + i * qcap;
      for (size_t k = 0; k < tmp.size() && k < (size_t)qcap; ++k) {
        q[k].key = tmp[k].x; q[k].id = tmp[k].y; q[k].t_arr = tmp[k].z;
        q[k].svc = (uint16_t)(tmp[k].w & 0xffff);
        q[k].budget = (int16_t)(tmp[k].w >> 16);
      }
    }
  }
  return IM_OK;
}

}  // extern "C"

// Validated restore of envs [env_begin, env_begin + env_count) and the tick;
// chain pools also take the chain words of queued and running calls and the
// pending calls (qch, sch, pend, pcount; NULL for single-call pools).
static im_status write_state_impl(im_pool* p, int32_t env_begin, int32_t env_count, int32_t tick,
                                  const im_env_state* envs, const im_model_state* models,
                                  const im_slot* slots, const im_entry* queues, const int64_t* hist,
                                  const im_chain* qch, const im_chain* sch, const im_pending* pend,
                                  const int32_t* pcount) {
  if (env_begin < 0 || env_count < 0 || (int64_t)env_begin + env_count > p->d.n_envs)
    return fail(p, IM_EINVAL, "env range out of bounds");
  if (!envs || !models || !slots || !queues || !hist) return fail(p, IM_EINVAL, "NULL argument");
  if (p->chains && (!qch || !sch || !pend || !pcount)) return fail(p, IM_EINVAL, "NULL argument");
  if (tick < 0) return fail(p, IM_EINVAL, "tick < 0");
  const bool ch = p->chains;
  // chain words: the call's query row, its index among n_steps calls, the
  // first call's role, the base service time and the query's budget
  auto chain_ok = [&](const im_chain& c) {
    return c.q_idx >= 0 && (int64_t)c.q_idx < p->Q && c.q_idx < (1 << 24) && c.n_steps >= 1 &&
           c.n_steps <= p->d.max_steps && c.k >= 0 && c.k < c.n_steps && c.base_svc >= 1 &&
           c.base_svc <= IM_SVC_MAX && c.beta >= 1 && c.beta <= 32767 && c.role0 >= 0 &&
           c.role0 < (p->d.net == IM_NET_DUAL ? p->d.n_roles : 1) && c.role0 < 32;
  };
  auto pack = [](const im_chain& c) {
    return make_int2(im::chain_a(c.q_idx, c.k, c.n_steps), im::chain_b(c.base_svc, c.beta, c.role0));
  };
  const int M = p->d.n_models, S = p->S, qcap = p->d.queue_cap, A = p->A;
  const size_t EMc = (size_t)env_count * M, em0 = (size_t)env_begin * M;
  std::vector<ModelRec> recs(EMc);
  std::memset(recs.data(), 0, EMc * sizeof(ModelRec));
  std::vector<int64_t> cnt(EMc * im::C_NUM, 0);
  std::vector<uint8_t> ring(EMc * im::kRpmRing, 0);
  std::vector<int4> fr(EMc * im::kFront, make_int4(0, 0, 0, 0));
  std::vector<int4> pl(EMc * (size_t)qcap, make_int4(0, 0, 0, 0));
  std::vector<int4> sl(EMc * S);
  std::vector<int2> frx(ch ? fr.size() : 0, make_int2(0, 0)), plx(ch ? pl.size() : 0, make_int2(0, 0)),
      slx(ch ? sl.size() : 0, make_int2(0, 0));
  for (size_t i = 0; i < EMc; ++i) {
    const im_model_state& ms = models[i];
    const int e = (int)(i / M);
    if (ms.qlen < 0 || ms.qlen > qcap || ms.capacity < 0 || ms.capacity > S || ms.ewma_q8 < 0)
      return fail(p, IM_ESTATE, "model state out of bounds");
    const im_entry* q = queues + i * qcap;
    int64_t bl = 0;
    for (int k = 0; k < ms.qlen; ++k) {
      bl += q[k].svc;
      if (k > 0 && !(q[k - 1].key < q[k].key || (q[k - 1].key == q[k].key && q[k - 1].id < q[k].id)))
        return fail(p, IM_ESTATE, "queue not strictly increasing in (key, id)");
      if (q[k].id < 0 || q[k].id >= envs[e].next_id) return fail(p, IM_ESTATE, "queue id out of range");
      // the schedule step recovers an entry's arrival tick from its key, budget
      // and service time, so the three must agree with the key mode
      if (q[k].svc < 1 || q[k].svc > IM_SVC_MAX * p->d.n_depths)
        return fail(p, IM_ESTATE, "queued service time out of range");
      // a chain's later call is queued with what is left of its query's budget (maybe <= 0)
      if (!ch && q[k].budget < 1) return fail(p, IM_ESTATE, "queued budget < 1");
      if (ch) {
        const im_chain& c = qch[i * qcap + k];
        if (!chain_ok(c) || q[k].svc % c.base_svc != 0 || q[k].svc / c.base_svc > p->d.n_depths)
          return fail(p, IM_ESTATE, "queued call's chain words out of range");
      }
      if (q[k].t_arr < 0 || q[k].t_arr >= tick) return fail(p, IM_ESTATE, "queued arrival tick out of range");
      const int64_t key = p->d.key_mode == IM_KEY_FCFS ? (int64_t)q[k].t_arr
                          : (p->d.key_mode == IM_KEY_DEADLINE ? (int64_t)q[k].t_arr + q[k].budget
                                                              : (int64_t)q[k].t_arr + q[k].budget - q[k].svc);
      if (key != q[k].key) return fail(p, IM_ESTATE, "queue key does not match t_arr, budget and svc");
    }
    if (bl != ms.backlog) return fail(p, IM_ESTATE, "backlog != sum of queued svc");
    int busy = 0, busy_mask = 0, next_done = INT32_MAX;
    for (int s = 0; s < S; ++s) {
      const im_slot& x = slots[i * S + s];
      if (x.id >= 0) {
        ++busy;
        if (x.rem < 1) return fail(p, IM_ESTATE, "busy slot with rem < 1");
        if (x.t_arr < 0 || x.t_arr >= tick || (!ch && x.budget < 1) || x.id >= envs[e].next_id)
          return fail(p, IM_ESTATE, "slot arrival tick, budget or id out of range");
        if (ch && !chain_ok(sch[i * S + s])) return fail(p, IM_ESTATE, "running call's chain words out of range");
        if ((int64_t)x.rem + tick - 1 > INT32_MAX) return fail(p, IM_ESTATE, "slot rem too large");
        busy_mask |= 1 << s;
        next_done = std::min(next_done, x.rem + tick - 1);
      }
      // device slot: {id, t_arr, completion tick, budget}
      sl[i * S + s] = x.id >= 0 ? make_int4(x.id, x.t_arr, x.rem + tick - 1, x.budget)
                                : make_int4(-1, 0, 0, 0);
      if (ch && x.id >= 0) slx[i * S + s] = pack(sch[i * S + s]);
    }
    if (busy != ms.busy) return fail(p, IM_ESTATE, "busy != occupied slots");
    ModelRec& r = recs[i];
    r.qlen = ms.qlen; r.busy = ms.busy; r.ewma = ms.ewma_q8; r.backlog = ms.backlog;
    r.cap = ms.capacity; r.enabled = ms.enabled ? 1 : 0; r.next_id = envs[e].next_id;
    r.t = tick;
    r.busy_mask = busy_mask;
    r.next_done = next_done;
    r.fh = 0;
    r.fn = std::min(ms.qlen, im::kFront);
    r.P = ms.qlen - r.fn;
    for (int k = 0; k < ms.qlen; ++k) {
      const int4 v = make_int4(q[k].key, q[k].id, q[k].t_arr,
                               (int32_t)((uint32_t)q[k].svc | ((uint32_t)q[k].budget << 16)));
      if (k < im::kFront) fr[i * im::kFront + k] = v;
      else pl[i * qcap + (k - im::kFront)] = v;
      if (ch) {
        const int2 x = pack(qch[i * qcap + k]);
        if (k < im::kFront) frx[i * im::kFront + k] = x;
        else plx[i * qcap + (k - im::kFront)] = x;
      }
    }
    int64_t* c = &cnt[i * im::C_NUM];
    c[im::C_REJ_OVERFLOW] = ms.rej_overflow; c[im::C_ENQUEUED] = ms.enqueued;
    c[im::C_STARTED] = ms.started; c[im::C_COMPLETED] = ms.completed; c[im::C_SLO_MET] = ms.slo_met;
    c[im::C_LAT_SUM] = ms.lat_sum; c[im::C_WAIT_SUM] = ms.wait_sum;
    c[im::C_COST_Q16] = ms.cost_q16;
    if (ms.rpm_limit < 0 || ms.rpm_limit > (1 << 30)) return fail(p, IM_ESTATE, "rpm_limit out of range");
    int hsum = 0;
    for (int k = 0; k < im::kRpmWindow; ++k) {
      hsum += ms.rpm_hist[k];
      if ((int64_t)tick - 1 - k >= 0)
        ring[i * im::kRpmRing + rpm_slot((int64_t)tick - 1 - k)] = ms.rpm_hist[k];
      else if (ms.rpm_hist[k] != 0)
        return fail(p, IM_ESTATE, "dispatches before tick 0");
    }
    if (hsum != ms.rpm_count) return fail(p, IM_ESTATE, "rpm_count != sum of rpm_hist");
    r.rpm_limit = ms.rpm_limit;
    r.rpm_count = ms.rpm_count;
    if (ms.rpm_limit > 0 || ms.rpm_count > 0) p->rpm_active = true;
    r.inv_rpm = ms.rpm_limit > 0 ? (float)(1.0 / ms.rpm_limit) : 0.f;
  }
  // pending calls, routed at the next tick: the buffer of parity `tick`
  const int PM = p->pend_cap;
  std::vector<int4> pr(ch ? (size_t)env_count * PM : 0, make_int4(0, 0, 0, 0));
  std::vector<int32_t> pcv(ch ? env_count : 0, 0);
  for (int e = 0; ch && e < env_count; ++e) {
    if (pcount[e] < 0 || pcount[e] > PM) return fail(p, IM_ESTATE, "pending count out of range");
    pcv[e] = pcount[e];
    for (int i = 0; i < pcount[e]; ++i) {
      const im_pending& x = pend[(size_t)e * PM + i];
      if (!chain_ok(x.ch) || x.ch.k < 1) return fail(p, IM_ESTATE, "pending call's chain words out of range");
      const int2 w = pack(x.ch);
      pr[(size_t)e * PM + i] = make_int4(w.x, w.y, x.deadline, 0);
    }
  }
  constexpr int EC = im::kEnvCnt;
  std::vector<int64_t> ec((size_t)env_count * EC);
  for (int e = 0; e < env_count; ++e) {
    ec[EC * e + im::E_ARRIVED] = envs[e].arrived;
    ec[EC * e + im::E_REJ_NOMODEL] = envs[e].rej_nomodel;
    ec[EC * e + im::E_Q_DONE] = envs[e].q_done;
    ec[EC * e + im::E_Q_MET] = envs[e].q_met;
  }
  IM_HIP(p, hipDeviceSynchronize());
  if (EMc) {
    IM_HIP(p, hipMemcpy(p->ms + em0, recs.data(), EMc * sizeof(ModelRec), hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->cnt + em0 * im::C_NUM, cnt.data(), cnt.size() * 8, hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->front + em0 * im::kFront, fr.data(), fr.size() * sizeof(int4), hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->qpool + em0 * qcap, pl.data(), pl.size() * sizeof(int4), hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->slots + em0 * S, sl.data(), sl.size() * sizeof(int4), hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->rpm_ring + em0 * im::kRpmRing, ring.data(), ring.size(), hipMemcpyHostToDevice));
    if (ch) {
      IM_HIP(p, hipMemcpy(p->front_ext + em0 * im::kFront, frx.data(), frx.size() * sizeof(int2), hipMemcpyHostToDevice));
      IM_HIP(p, hipMemcpy(p->pool_ext + em0 * qcap, plx.data(), plx.size() * sizeof(int2), hipMemcpyHostToDevice));
      IM_HIP(p, hipMemcpy(p->slot_ext + em0 * S, slx.data(), slx.size() * sizeof(int2), hipMemcpyHostToDevice));
    }
  }
  if (ch && env_count) {
    const size_t par = (size_t)(tick & 1), E = p->d.n_envs;
    IM_HIP(p, hipMemcpy(p->pcnt + par * E + env_begin, pcv.data(), pcv.size() * 4, hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->pend + (par * E + env_begin) * PM, pr.data(), pr.size() * sizeof(int4),
                        hipMemcpyHostToDevice));
  }
  if (env_count) {
    IM_HIP(p, hipMemcpy(p->env_cnt + (size_t)env_begin * EC, ec.data(), ec.size() * 8, hipMemcpyHostToDevice));
    IM_HIP(p, hipMemcpy(p->hist + (size_t)env_begin * A, hist, (size_t)env_count * A * 8, hipMemcpyHostToDevice));
  }
  IM_HIP(p, im::launch_snapshot(sched_args(p), env_begin, env_count, nullptr));
  IM_HIP(p, hipDeviceSynchronize());
  p->t = tick;
  return IM_OK;
}

extern "C" {

im_status im_write_state(im_pool* p, int32_t env_begin, int32_t env_count, int32_t tick,
                         const im_env_state* envs, const im_model_state* models,
                         const im_slot* slots, const im_entry* queues, const int64_t* hist) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (p->chains) return fail(p, IM_EUNSUPPORTED, "im_write_state: chain pools restore with im_write_chain_state");
  return write_state_impl(p, env_begin, env_count, tick, envs, models, slots, queues, hist, nullptr, nullptr,
                          nullptr, nullptr);
}

im_status im_write_chain_state(im_pool* p, int32_t env_begin, int32_t env_count, int32_t tick,
                               const im_env_state* envs, const im_model_state* models,
                               const im_slot* slots, const im_entry* queues, const int64_t* hist,
                               const im_chain* queue_chains, const im_chain* slot_chains,
                               const im_pending* pending, const int32_t* pending_count) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (!p->chains) return fail(p, IM_EINVAL, "im_write_chain_state: not a chain pool");
  return write_state_impl(p, env_begin, env_count, tick, envs, models, slots, queues, hist, queue_chains,
                          slot_chains, pending, pending_count);
}

im_status im_read_chain_state(im_pool* p, int32_t env_begin, int32_t env_count, im_chain* queues,
                              im_chain* slots, im_pending* pending, int32_t* pending_count) {
  if (!p) return fail(nullptr, IM_EINVAL, "pool is NULL");
  if (!p->chains) return fail(p, IM_EINVAL, "im_read_chain_state: not a chain pool");
  if (env_begin < 0 || env_count < 0 || (int64_t)env_begin + env_count > p->d.n_envs)
    return fail(p, IM_EINVAL, "env range out of bounds");
  IM_HIP(p, hipDeviceSynchronize());
  const int M = p->d.n_models, S = p->S, qcap = p->d.queue_cap, PM = p->pend_cap;
  const size_t em0 = (size_t)env_begin * M, EMc = (size_t)env_count * M, E = p->d.n_envs;
  if (EMc == 0) return IM_OK;
  std::vector<ModelRec> recs(EMc);
  IM_HIP(p, hipMemcpy(recs.data(), p->ms + em0, EMc * sizeof(ModelRec), hipMemcpyDeviceToHost));
  const int32_t t = recs[0].t;
  auto unpack = [](int2 x) {
    im_chain c;
    c.q_idx = im::chain_q(x.x);
    c.k = (int16_t)im::chain_k(x.x);
    c.n_steps = (int16_t)im::chain_n(x.x);
    c.role0 = (int16_t)im::chain_role0(x.y);
    c.base_svc = (int16_t)im::chain_base(x.y);
    c.beta = im::chain_beta(x.y);
    return c;
  };
  if (queues) {
    // the same service order as im_read_state: the front, then the pool by (key, id)
    std::vector<int4> fr(EMc * im::kFront), pl(EMc * (size_t)qcap);
    std::vector<int2> frx(fr.size()), plx(pl.size());
    IM_HIP(p, hipMemcpy(fr.data(), p->front + em0 * im::kFront, fr.size() * sizeof(int4), hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(frx.data(), p->front_ext + em0 * im::kFront, frx.size() * sizeof(int2), hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(pl.data(), p->qpool + em0 * qcap, pl.size() * sizeof(int4), hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(plx.data(), p->pool_ext + em0 * qcap, plx.size() * sizeof(int2), hipMemcpyDeviceToHost));
    std::memset(queues, 0, EMc * qcap * sizeof(im_chain));
    std::vector<std::pair<int4, int2>> tmp;
    for (size_t i = 0; i < EMc; ++i) {
      const ModelRec& r = recs[i];
      tmp.clear();
      for (int k = r.fh; k < r.fh + r.fn; ++k) tmp.push_back({fr[i * im::kFront + k], frx[i * im::kFront + k]});
      const size_t f = tmp.size();
      for (int k = 0; k < r.P; ++k) tmp.push_back({pl[i * qcap + k], plx[i * qcap + k]});
      std::sort(tmp.begin() + f, tmp.end(), [](const std::pair<int4, int2>& x, const std::pair<int4, int2>& y) {
        return x.first.x != y.first.x ? x.first.x < y.first.x : x.first.y < y.first.y;
      });
      for (size_t k = 0; k < tmp.size() && k < (size_t)qcap; ++k) queues[i * qcap + k] = unpack(tmp[k].second);
    }
  }
  if (slots) {
    std::vector<int4> sl(EMc * S);
    std::vector<int2> slx(EMc * S);
    IM_HIP(p, hipMemcpy(sl.data(), p->slots + em0 * S, sl.size() * sizeof(int4), hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(slx.data(), p->slot_ext + em0 * S, slx.size() * sizeof(int2), hipMemcpyDeviceToHost));
    for (size_t i = 0; i < sl.size(); ++i) {
      if (sl[i].x >= 0) slots[i] = unpack(slx[i]);
      else std::memset(&slots[i], 0, sizeof(im_chain));
    }
  }
  if (pending || pending_count) {
    // the pending calls of the next tick: the buffer of parity t
    std::vector<int32_t> pc(env_count);
    std::vector<int4> pr((size_t)env_count * PM);
    const size_t par = (size_t)(t & 1);
    IM_HIP(p, hipMemcpy(pc.data(), p->pcnt + par * E + env_begin, pc.size() * 4, hipMemcpyDeviceToHost));
    IM_HIP(p, hipMemcpy(pr.data(), p->pend + (par * E + env_begin) * PM, pr.size() * sizeof(int4),
                        hipMemcpyDeviceToHost));
    for (int e = 0; e < env_count; ++e) {
      if (pending_count) pending_count[e] = pc[e];
      if (!pending) continue;
      for (int i = 0; i < PM; ++i) {
        im_pending& o = pending[(size_t)e * PM + i];
        if (i < pc[e]) {
          const int4 v = pr[(size_t)e * PM + i];
          o.ch = unpack(make_int2(v.x, v.y));
          o.deadline = v.z;
        } else {
          std::memset(&o, 0, sizeof(o));
        }
      }
    }
  }
  return IM_OK;
}

}  // extern "C"
