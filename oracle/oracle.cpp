// Oracle of the batched route-and-schedule tick.
//
// TEST INFRASTRUCTURE ONLY. This is the plain, slow, scalar CPU definition
// that the GPU library is checked against. Only the tests, the smoke check and
// the CPU-baseline leg of the benchmark may load it. It shares no source,
// header, table or constant generator with the GPU library.
//
// What it computes (per independent env e, per tick t), following the paper:
//   Sec. 3 "State" (Eq. 1): the executor observes the query embedding, the
//     remaining budget and per-model queue depth, latency and KV-cache load.
//   Sec. 3 "Action": a joint action a in [0, N*|S|) decodes to model a / K and
//     reasoning depth a % K.
//   Sec. 4.2: a policy network scores every joint action and is deployed
//     greedily (masked argmax): either a plain MLP over the state vector or
//     the paper's dual-pathway executor (a semantic pathway over the query
//     and role embeddings, a resource pathway over the remaining budget and
//     the per-model load, each ending in a LayerNorm, merged into one
//     representation that feeds the action and value heads). For RL rollouts (Sec. 4.4, Eq. 5 consumes
//     log pi, the entropy and V) the policy pi(a|s) is the softmax of the
//     logits over the valid actions, sampled with the Gumbel-max trick from
//     Philox4x32-10 noise (Salmon et al., SC 2011), and an optional value row
//     V(s) = w_val . h + b_val shares the last hidden layer h (Sec. 4.2
//     "Decision").
//   Sec. 4.3: every model's queue is served earliest-deadline-first with the
//     deadline t_arrive + budget; the default key is the latest start time
//     (deadline - service time), i.e. the slack.
//   Sec. 5.4: the latency signal is an exponential moving average of observed
//     end-to-end latency.
//   Table 5: each model serves a bounded number of sequences at once.
// Where the paper is silent, the readings are the documented ones: integer
// ticks, c_m concurrent service slots, ties broken by request id, tail-drop
// admission, alpha = 1/8 Q8 fixed-point EWMA, features normalised by
// reciprocals rounded once to fp32.
//
// Parity status: pinned by the golden example, closed-form invariants, a
// textbook single-server simulator, brute force over forced actions and
// library routines (see tests). The policy arithmetic is in fp64.

#include <algorithm>
#include <cfenv>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <thread>
#include <vector>

namespace {

// ----- limits of the boundary the oracle mirrors --------------------------
const int kSvcMax = 4095;      // base service time must lie in [1, kSvcMax]
const int kRpmWindow = 60;     // App. C: 60-second (tick) sliding window of dispatches

enum ErrBits {
  ERR_QIDX = 1,      // q_idx outside [0, Q)
  ERR_COUNT = 2,     // offsets not a valid CSR or n_e > max arrivals
  ERR_BUDGET = 4,    // budget < 1
  ERR_SVC = 8,       // base_svc outside [1, kSvcMax]
  ERR_ACTION = 16,   // action outside [-1, A)
  ERR_ROLE = 32,     // role outside [0, n_roles) (dual-pathway executor only)
  ERR_STEPS = 64,    // n_steps outside [1, max_steps] (multi-step chains only)
};

// ----- bf16 round-to-nearest-even of a real value ------------------------
// bf16 keeps 8 significant bits and fp32's exponent range (normal numbers
// down to 2^-126, subnormal quantum 2^-133). Round |v| to the nearest
// multiple of its quantum, ties to even (the default FE_TONEAREST mode).
double round_bf16(double v) {
  if (v == 0.0 || !std::isfinite(v)) return v;
  int e;
  std::frexp(v, &e);                        // v = f * 2^e with 0.5 <= |f| < 1
  int qexp = std::max(e - 8, -133);         // quantum of the bf16 grid at v
  double r = std::nearbyint(std::ldexp(v, -qexp));
  double out = std::ldexp(r, qexp);
  const double kMax = std::ldexp(255.0, 120);  // largest finite bf16 (1.9921875 * 2^127)
  if (std::fabs(out) > kMax) return std::copysign(INFINITY, v);
  return out;
}

// ----- data -----------------------------------------------------------------
// The query a call belongs to (multi-step chains; a single-step request is
// a query of one call): its embedding row, the call's index k among the
// query's n_steps sequential calls, the role of its first call, the base
// service time of every call and the query's budget beta.
struct Chain {
  int32_t q_idx = 0, k = 0, n_steps = 1, role0 = 0, base = 0, beta = 0;
};

struct Entry {            // a queued request (one call)
  int32_t key;            // sort key (slack / deadline / arrival tick)
  int32_t id;             // per-env request id, increasing in arrival order
  int32_t t_arr;          // tick the call entered the queue
  int32_t svc;            // service time in ticks = base_svc * (depth + 1)
  int32_t budget;         // time budget in ticks (a later call: what is left of the query's)
  Chain ch;
};

struct Slot {             // a service slot of a model
  bool busy = false;
  int32_t id = -1, t_arr = 0, rem = 0, budget = 0;
  Chain ch;
};

// A call spawned by the completion of the previous call of its query, routed
// at the next tick with the query's deadline.
struct Pending {
  Chain ch;
  int32_t deadline;
};

struct ModelState {
  std::vector<Entry> queue;   // sorted by key, ties by id (head = index 0)
  std::vector<Slot> slots;    // max_slots slots, only s < cap are filled
  int32_t ewma_q8 = 0;        // latency EWMA in Q8 fixed point (ticks * 256)
  int64_t backlog = 0;        // sum of svc over the queue
  int32_t cap = 0;            // c_m, concurrent service slots
  int32_t enabled = 1;
  int64_t rej_overflow = 0, enqueued = 0, started = 0, completed = 0,
          slo_met = 0, lat_sum = 0, wait_sum = 0;
  int64_t cost_q16 = 0;       // sum over completions of floor(2^16 latency / budget)
  // Blackbox proxy (Sec. 5.5, App. C): with rpm_limit > 0 the model is an API
  // behind a rate limit; every dispatch (a request entering a service slot)
  // is timestamped, and a request is dispatched only while fewer than
  // rpm_limit dispatches fall in the last kRpmWindow ticks.
  int32_t rpm_limit = 0;
  std::vector<int32_t> dispatch_ticks;
};

// Dispatches of a model at ticks in (t_end - kRpmWindow, t_end].
int rpm_count(const ModelState& ms, int32_t t_end) {
  int n = 0;
  for (int32_t tau : ms.dispatch_ticks) n += (tau > t_end - kRpmWindow && tau <= t_end) ? 1 : 0;
  return n;
}

struct EnvState {
  std::vector<ModelState> models;
  int32_t next_id = 0;
  int64_t arrived = 0, rej_nomodel = 0;
  std::vector<int64_t> hist;  // routed requests per joint action
  std::vector<Pending> pending;      // calls to route at the next tick, in spawn order
  int64_t q_done = 0, q_met = 0;     // chains: queries whose last call completed / on time
};

}  // namespace

extern "C" {

// Pool description (the oracle's own struct; field order is its own).
struct orc_desc {
  int32_t E, M, K, qcap, max_slots, embed_dim, feat_dim, n_layers;
  int32_t widths[4];
  int32_t dtype;          // 0 fp32, 1 bf16 (weights, inputs, hidden rounded)
  int32_t key_mode;       // 0 slack, 1 deadline, 2 fcfs
  int32_t max_arrivals;
  int32_t budget_max;
  int32_t value_head;     // 1: the last layer has M*K + 1 rows, row M*K is V(s)
  int32_t net;            // 0 plain MLP, 1 dual-pathway executor (Sec. 4.2)
  int32_t n_roles;        // dual-pathway executor: rows of the role-embedding table
  int32_t max_steps;      // > 1: multi-step agent chains (calls per query up to this)
  int64_t Q;
};

// Parameters of the dual-pathway executor (Sec. 4.2), matrices [out x in]
// row-major. In bf16 pools the matrices and the role table hold bf16 values.
struct orc_dual {
  std::vector<double> W_sem, b_sem, g_sem, be_sem;   // 128 x 2 E_d; LayerNorm gain, bias
  std::vector<double> W_bud, b_bud;                  // 16 x 1
  std::vector<double> W_sys, b_sys;                  // 16 x 3M, input [queue | e2e | kv]
  std::vector<double> W_res, b_res, g_res, be_res;   // 64 x 32, input [h_bud | h_sys]
  std::vector<double> W_merge, b_merge;              // 128 x 192, input [h_sem | h_res]
  std::vector<double> W_act, b_act;                  // (M K + value_head) x 128
  std::vector<double> role;                          // n_roles x E_d
};

struct orc_pool {
  orc_desc d;
  int A;
  std::vector<std::vector<double>> W;   // [layer] out x in, row-major
  std::vector<std::vector<double>> b;   // [layer] out
  orc_dual dual;                        // the dual-pathway executor (net == 1)
  std::vector<float> emb;               // Q x embed_dim (value of each entry)
  std::vector<double> logit_bias;       // M (0 when absent)
  std::vector<EnvState> envs;
  int32_t t = 0;
  int32_t err = 0;
  int64_t dual_completed = 0, dual_cost_q16 = 0;   // totals at the last dual update
  // chain pools: the arrival CSR of the current call starts at 0, never
  // decreases and ends at n_total (set by each entry point that reads it)
  mutable bool csr_whole = true;
};

}  // extern "C"

namespace {

// Feature vector of one request (Eq. 1 restated for the build):
//   [ emb[q_idx] | qlen_m/QCAP | busy_m/c_m | ewma_m/(256 B) | backlog_m/(c_m B) |
//     budget/B | 0 ... ]
// with B = budget_max, stats laid out stat-major (all models' queue depth,
// then all models' KV proxy, ...). Every reciprocal is computed in fp64 and
// rounded once to fp32; each feature is one fp32 product. In bf16 pools the
// vector is then rounded to bf16.
void features(const orc_pool* p, const EnvState& env, int32_t q_idx, int32_t budget,
              std::vector<double>& x) {
  const orc_desc& d = p->d;
  const int M = d.M;
  x.assign(d.feat_dim, 0.0);
  for (int k = 0; k < d.embed_dim; ++k)
    x[k] = p->emb[(size_t)q_idx * d.embed_dim + k];
  const float inv_qcap = (float)(1.0 / d.qcap);
  const float inv_lat = (float)(1.0 / (256.0 * d.budget_max));
  const float inv_bud = (float)(1.0 / d.budget_max);
  for (int m = 0; m < M; ++m) {
    const ModelState& ms = env.models[m];
    int busy = 0;
    for (const Slot& s : ms.slots) busy += s.busy ? 1 : 0;
    const int c = std::max(ms.cap, 1);
    const float inv_c = (float)(1.0 / c);
    const float inv_clat = (float)(1.0 / ((double)c * d.budget_max));
    // queue-depth signal: recent dispatches / RPM limit for a blackbox model
    // (Sec. 5.5), the queue depth / QCAP otherwise; the window ends at the
    // last completed tick (the route step reads the state after it)
    float f_q = ms.rpm_limit > 0 ? (float)rpm_count(ms, p->t - 1) * (float)(1.0 / ms.rpm_limit)
                                 : (float)ms.queue.size() * inv_qcap;
    float f_kv = (float)busy * inv_c;
    float f_lat = (float)ms.ewma_q8 * inv_lat;
    float f_bl = (float)ms.backlog * inv_clat;
    x[d.embed_dim + 0 * M + m] = f_q;
    x[d.embed_dim + 1 * M + m] = f_kv;
    x[d.embed_dim + 2 * M + m] = f_lat;
    x[d.embed_dim + 3 * M + m] = f_bl;
  }
  float f_b = (float)budget * inv_bud;
  x[d.embed_dim + 4 * M] = f_b;
  if (d.dtype == 1)
    for (double& v : x) v = round_bf16(v);
}

// Policy MLP in fp64: hidden layers ReLU(W h + b), output W h + b, then the
// per-model logit bias. In bf16 pools every hidden activation is rounded to
// bf16 after the ReLU (weights were rounded at creation).
void mlp(const orc_pool* p, const std::vector<double>& x, std::vector<double>& z) {
  std::vector<double> h = x, y;
  const int L = p->d.n_layers;
  for (int l = 0; l < L; ++l) {
    const int out = p->d.widths[l];
    const int in = (int)h.size();
    y.assign(out, 0.0);
    for (int o = 0; o < out; ++o) {
      double s = p->b[l][o];
      for (int i = 0; i < in; ++i) s += p->W[l][(size_t)o * in + i] * h[i];
      y[o] = s;
    }
    if (l + 1 < L) {
      for (double& v : y) {
        v = v > 0.0 ? v : 0.0;
        if (p->d.dtype == 1) v = round_bf16(v);
      }
    }
    h.swap(y);
  }
  z = h;
  for (int a = 0; a < p->A; ++a) z[a] += p->logit_bias[a / p->d.K];
}

// ----- the paper's dual-pathway executor (Sec. 4.2) -------------------------
// Widths fixed by the paper: semantic pathway 128, budget and system heads 16
// each, resource pathway 64, merged representation 128.
const int kSem = 128, kBud = 16, kSys = 16, kRes = 64, kMerge = 128;
// LayerNorm: the paper gives no epsilon; 1e-5 (the usual default) is taken.
const double kLnEps = 1e-5;

// y = W x + b for W [out x in] row-major.
void linear(const std::vector<double>& W, const std::vector<double>& b, int out,
            const std::vector<double>& x, std::vector<double>& y) {
  const size_t in = x.size();
  y.assign(out, 0.0);
  for (int o = 0; o < out; ++o) {
    double s = b[o];
    for (size_t i = 0; i < in; ++i) s += W[(size_t)o * in + i] * x[i];
    y[o] = s;
  }
}

void relu_inplace(std::vector<double>& v) {
  for (double& x : v) x = x > 0.0 ? x : 0.0;
}

// LayerNorm over the whole vector: (v - mean) / sqrt(var + eps) * gain + bias,
// with the biased (1/n) variance.
void layer_norm(std::vector<double>& v, const std::vector<double>& gain,
                const std::vector<double>& bias) {
  const double n = (double)v.size();
  double mean = 0.0;
  for (double x : v) mean += x;
  mean /= n;
  double var = 0.0;
  for (double x : v) var += (x - mean) * (x - mean);
  var /= n;
  const double inv = 1.0 / std::sqrt(var + kLnEps);
  for (size_t i = 0; i < v.size(); ++i) v[i] = (v[i] - mean) * inv * gain[i] + bias[i];
}

// Hidden vectors of one request through the dual-pathway executor, in fp64.
// x is the request's feature vector (features()): query embedding, the four
// per-model load statistics (stat-major: queue depth, KV proxy, latency,
// backlog) and the normalised remaining budget, already bf16 in bf16 pools.
// In bf16 pools every vector that enters a matrix product is bf16: h_bud and
// h_sys after their ReLU, h_sem and h_res after their LayerNorm, h after its
// ReLU (the weights were rounded at creation).
struct DualTrace {
  std::vector<double> h_sem, h_bud, h_sys, h_res, h, z;
};

void dual_net(const orc_pool* p, const std::vector<double>& x, int32_t role, DualTrace& t) {
  const orc_desc& d = p->d;
  const orc_dual& w = p->dual;
  const int Ed = d.embed_dim, M = d.M;
  auto rnd = [&](std::vector<double>& v) {
    if (d.dtype == 1) for (double& a : v) a = round_bf16(a);
  };
  // semantic pathway: LN(ReLU(W_sem [e_q | e_r]))
  std::vector<double> sem_in(2 * Ed);
  for (int k = 0; k < Ed; ++k) sem_in[k] = x[k];
  for (int k = 0; k < Ed; ++k) sem_in[Ed + k] = w.role[(size_t)role * Ed + k];
  linear(w.W_sem, w.b_sem, kSem, sem_in, t.h_sem);
  relu_inplace(t.h_sem);
  layer_norm(t.h_sem, w.g_sem, w.be_sem);
  rnd(t.h_sem);
  // resource pathway: budget head over b, system head over
  // [queue depth | end-to-end latency | KV-cache use] of every model
  const std::vector<double> b_in = {x[Ed + 4 * M]};
  linear(w.W_bud, w.b_bud, kBud, b_in, t.h_bud);
  relu_inplace(t.h_bud);
  rnd(t.h_bud);
  std::vector<double> sys_in(3 * M);
  for (int m = 0; m < M; ++m) {
    sys_in[m] = x[Ed + 0 * M + m];           // queue depth
    sys_in[M + m] = x[Ed + 2 * M + m];       // end-to-end latency
    sys_in[2 * M + m] = x[Ed + 1 * M + m];   // KV-cache use
  }
  linear(w.W_sys, w.b_sys, kSys, sys_in, t.h_sys);
  relu_inplace(t.h_sys);
  rnd(t.h_sys);
  std::vector<double> res_in(t.h_bud);
  res_in.insert(res_in.end(), t.h_sys.begin(), t.h_sys.end());
  linear(w.W_res, w.b_res, kRes, res_in, t.h_res);
  relu_inplace(t.h_res);
  layer_norm(t.h_res, w.g_res, w.be_res);
  rnd(t.h_res);
  // decision: h = ReLU(W_merge [h_sem | h_res]); logits W_act h (+ value row)
  std::vector<double> mrg_in(t.h_sem);
  mrg_in.insert(mrg_in.end(), t.h_res.begin(), t.h_res.end());
  linear(w.W_merge, w.b_merge, kMerge, mrg_in, t.h);
  relu_inplace(t.h);
  rnd(t.h);
  linear(w.W_act, w.b_act, p->A + d.value_head, t.h, t.z);
}

// Logits of one request (rows A.. hold the value head), with the per-model
// logit bias on the action rows.
void policy(const orc_pool* p, const EnvState& env, int32_t q_idx, int32_t role, int32_t budget,
            std::vector<double>& z) {
  std::vector<double> x;
  features(p, env, q_idx, budget, x);
  if (p->d.net == 1) {
    DualTrace t;
    dual_net(p, x, role, t);
    z = t.z;
    for (int a = 0; a < p->A; ++a) z[a] += p->logit_bias[a / p->d.K];
  } else {
    mlp(p, x, z);
  }
}

// Role of row r: 0 for MLP pools; -1 when out of range or missing.
int32_t role_of(const orc_pool* p, const int16_t* role, int32_t r) {
  if (p->d.net != 1) return 0;
  if (!role || role[r] < 0 || role[r] >= p->d.n_roles) return -1;
  return role[r];
}

bool model_valid(const orc_pool* p, const ModelState& ms) {
  return ms.enabled != 0 && ms.cap > 0 && (int)ms.queue.size() < p->d.qcap;
}

int32_t sort_key(const orc_pool* p, int32_t t, int32_t budget, int32_t svc) {
  const int32_t deadline = t + budget;          // Sec. 4.3: t_arrive + beta
  switch (p->d.key_mode) {
    case 1: return deadline;                    // EDF by deadline
    case 2: return t;                           // FCFS
    default: return deadline - svc;             // latest start time (slack)
  }
}

// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as
// easy as 1, 2, 3", SC 2011): ten rounds of two 32x32->64-bit multiplies by
// the round multipliers, the high halves xored with the other two counter
// words and the key; the key is bumped by the Weyl constants between rounds.
void philox4x32_10(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  const uint64_t kMul0 = 0xD2511F53u, kMul1 = 0xCD9E8D57u;
  const uint32_t kWeyl0 = 0x9E3779B9u, kWeyl1 = 0xBB67AE85u;
  uint32_t c[4] = {ctr_in[0], ctr_in[1], ctr_in[2], ctr_in[3]};
  uint32_t k[2] = {key_in[0], key_in[1]};
  for (int round = 0; round < 10; ++round) {
    if (round > 0) { k[0] += kWeyl0; k[1] += kWeyl1; }
    const uint64_t p0 = kMul0 * (uint64_t)c[0];
    const uint64_t p1 = kMul1 * (uint64_t)c[2];
    const uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
    const uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
    const uint32_t n0 = hi1 ^ c[1] ^ k[0];
    const uint32_t n2 = hi0 ^ c[3] ^ k[1];
    c[0] = n0; c[1] = lo1; c[2] = n2; c[3] = lo0;
  }
  for (int i = 0; i < 4; ++i) out[i] = c[i];
}

// Uniform in (0, 1) from a 32-bit word: its top 23 bits plus one half, times
// 2^-23 (exact in fp32 and fp64, never 0 or 1).
double uniform23(uint32_t x) { return ((double)(x >> 9) + 0.5) * (1.0 / 8388608.0); }

// Gumbel noise of joint action a of request `id` of env `env`: word a % 4 of
// the Philox block with counter (id, env, a / 4, 0) and key (seed_lo, seed_hi).
double gumbel(uint32_t seed_lo, uint32_t seed_hi, int32_t id, int32_t env, int a) {
  const uint32_t ctr[4] = {(uint32_t)id, (uint32_t)env, (uint32_t)(a / 4), 0u};
  const uint32_t key[2] = {seed_lo, seed_hi};
  uint32_t w[4];
  philox4x32_10(ctr, key, w);
  const double u = uniform23(w[a % 4]);
  return -std::log(-std::log(u));
}

// ----- the rows of one env at one tick ---------------------------------------
// Multi-step chains (Sec. 4.3, Fig. 3): a query of n_steps calls runs them in
// sequence; the completion of call k spawns call k + 1, routed at the next
// tick. Every call inherits the query's deadline t_arrive + beta: a call
// routed at tick t has the remaining budget deadline - t. An env's rows at a
// tick are its pending calls in spawn order, then its new arrivals in
// arrival order; request ids follow that order. Single-step pools have no
// pending calls and their rows are the arrivals.
struct Row {
  int32_t out;        // index of the row's outputs (actions, logits, ...)
  int32_t src;        // arrival row, or -1 for a pending call
  int32_t q_idx, role, budget, base_svc;   // role of this call; budget: what is left
  Chain ch;
};

bool chains(const orc_pool* p) { return p->d.max_steps > 1; }

// Chain pools lay an env's rows out by a scan over the arrival CSR, after the
// pending calls of the envs before it. Reading: a CSR that is not one
// monotone partition of [0, n_total) makes no arrival usable; every env then
// skips the tick with ERR_COUNT (its pending calls stay pending).
void set_csr_whole(const orc_pool* p, int32_t n_total, const int32_t* off) {
  bool w = off[0] == 0 && off[p->d.E] == n_total;
  for (int e = 0; w && e < p->d.E; ++e) w = off[e + 1] >= off[e];
  p->csr_whole = w;
}

// Arrival CSR entry of env e usable (chain pools route only such arrivals).
bool csr_ok(const orc_pool* p, int e, int32_t n_total, const int32_t* off) {
  if (chains(p) && !p->csr_whole) return false;
  const int32_t lo = off[e], hi = off[e + 1];
  return lo >= 0 && hi >= lo && hi <= n_total && hi - lo <= p->d.max_arrivals;
}

// Start of env e's rows in the output arrays: the arrival offsets for
// single-step pools; for chain pools the running sum over the envs before e
// of their pending calls and usable arrivals.
std::vector<int32_t> row_offsets(const orc_pool* p, int32_t n_total, const int32_t* off) {
  std::vector<int32_t> o(p->d.E + 1, 0);
  if (!chains(p)) {
    for (int e = 0; e <= p->d.E; ++e) o[e] = off[e];
    return o;
  }
  for (int e = 0; e < p->d.E; ++e)
    o[e + 1] = o[e] + (int32_t)p->envs[e].pending.size() +
               (csr_ok(p, e, n_total, off) ? off[e + 1] - off[e] : 0);
  return o;
}

int32_t clamp16(int64_t v) { return (int32_t)std::max<int64_t>(-32768, std::min<int64_t>(32767, v)); }

std::vector<Row> env_rows(const orc_pool* p, int e, int32_t n_total, const int32_t* off,
                          const std::vector<int32_t>& ro, const int32_t* q_idx,
                          const int16_t* role, const int16_t* budget, const int16_t* base_svc,
                          const int16_t* n_steps) {
  std::vector<Row> rows;
  const EnvState& env = p->envs[e];
  int32_t out = ro[e];
  for (const Pending& pd : env.pending) {
    Row r;
    r.out = out++;
    r.src = -1;
    r.ch = pd.ch;
    r.q_idx = pd.ch.q_idx;
    r.role = p->d.net == 1 ? (pd.ch.role0 + pd.ch.k) % p->d.n_roles : 0;
    r.budget = clamp16((int64_t)pd.deadline - p->t);
    r.base_svc = pd.ch.base;
    rows.push_back(r);
  }
  if (chains(p) && !csr_ok(p, e, n_total, off)) return rows;
  for (int32_t i = off[e]; i < off[e + 1]; ++i) {
    Row r;
    r.out = chains(p) ? out++ : i;
    r.src = i;
    r.q_idx = q_idx[i];
    r.role = role_of(p, role, i);
    r.budget = budget[i];
    r.base_svc = base_svc ? base_svc[i] : 1;
    r.ch.q_idx = q_idx[i];
    r.ch.k = 0;
    r.ch.n_steps = chains(p) ? (n_steps ? n_steps[i] : 1) : 1;
    r.ch.role0 = r.role < 0 ? 0 : r.role;
    r.ch.base = r.base_svc;
    r.ch.beta = budget[i];
    rows.push_back(r);
  }
  return rows;
}

// Route the rows of env e: logits (post-bias, pre-mask) and actions.
void route_env(orc_pool* p, int e, const std::vector<Row>& rows, double* logits,
               int32_t* actions, int32_t* err) {
  const EnvState& env = p->envs[e];
  std::vector<double> z;
  for (const Row& r : rows) {
    const bool bad_q = r.q_idx < 0 || (int64_t)r.q_idx >= p->d.Q;
    if (bad_q || r.role < 0) {
      if (bad_q) *err |= ERR_QIDX;
      if (r.role < 0) *err |= ERR_ROLE;
      actions[r.out] = -1;
      if (logits) for (int a = 0; a < p->A; ++a) logits[(size_t)r.out * p->A + a] = 0.0;
      continue;
    }
    policy(p, env, r.q_idx, r.role, r.budget, z);
    int best = -1;
    for (int a = 0; a < p->A; ++a) {
      const ModelState& ms = env.models[a / p->d.K];
      if (!model_valid(p, ms)) continue;
      if (best < 0 || z[a] > z[best]) best = a;   // strict: lowest index wins ties
    }
    actions[r.out] = best;
    if (logits) for (int a = 0; a < p->A; ++a) logits[(size_t)r.out * p->A + a] = z[a];
  }
}

// RL-rollout route of env e (global index env_base + e): besides the logits,
// the action drawn from pi(.|s) = softmax of the logits over the valid actions
// (Gumbel-max: argmax over valid a of z_a + G_a, lowest index on ties) or, if
// greedy, the masked argmax; log pi of that action; the entropy of pi; and
// the value row. No valid action: action -1, log-prob 0, entropy 0.
void route_env_rl(orc_pool* p, int e, int env_base, const std::vector<Row>& rows,
                  uint32_t seed_lo, uint32_t seed_hi, int greedy, double* logits,
                  int32_t* actions, double* logp, double* entropy, double* value, int32_t* err) {
  const EnvState& env = p->envs[e];
  const int A = p->A;
  std::vector<double> z;
  for (size_t i = 0; i < rows.size(); ++i) {
    const Row& r = rows[i];
    const int32_t o = r.out;
    const bool bad_q = r.q_idx < 0 || (int64_t)r.q_idx >= p->d.Q;
    if (bad_q || r.role < 0) {
      if (bad_q) *err |= ERR_QIDX;
      if (r.role < 0) *err |= ERR_ROLE;
      actions[o] = -1;
      logp[o] = 0.0; entropy[o] = 0.0; value[o] = 0.0;
      if (logits) for (int a = 0; a < A; ++a) logits[(size_t)o * A + a] = 0.0;
      continue;
    }
    policy(p, env, r.q_idx, r.role, r.budget, z);
    value[o] = p->d.value_head ? z[A] : 0.0;
    if (logits) for (int a = 0; a < A; ++a) logits[(size_t)o * A + a] = z[a];
    std::vector<int> valid;
    for (int a = 0; a < A; ++a)
      if (model_valid(p, env.models[a / p->d.K])) valid.push_back(a);
    if (valid.empty()) {
      actions[o] = -1; logp[o] = 0.0; entropy[o] = 0.0;
      continue;
    }
    // log-sum-exp over the valid actions, shifted by their largest logit
    double zmax = z[valid[0]];
    for (int a : valid) zmax = std::max(zmax, z[a]);
    double sum = 0.0;
    for (int a : valid) sum += std::exp(z[a] - zmax);
    const double lse = zmax + std::log(sum);
    double h = 0.0;                         // -sum pi log pi
    for (int a : valid) {
      const double lp = z[a] - lse;
      h -= std::exp(lp) * lp;
    }
    const int32_t id = env.next_id + (int32_t)i;
    int best = -1;
    double best_score = 0.0;
    for (int a : valid) {
      const double sc = greedy ? z[a] : z[a] + gumbel(seed_lo, seed_hi, id, env_base + e, a);
      if (best < 0 || sc > best_score) { best = a; best_score = sc; }
    }
    actions[o] = best;
    logp[o] = z[best] - lse;
    entropy[o] = h;
  }
}

// Admission, queue insertion, service and accounting for env e at tick t.
void schedule_env(orc_pool* p, int e, int32_t n_total, const int32_t* off,
                  const std::vector<Row>& rows, const int32_t* actions, int32_t* err) {
  const orc_desc& d = p->d;
  EnvState& env = p->envs[e];
  // Validate the whole env first; an invalid env is left untouched this tick
  // (its pending calls stay pending).
  int bad = 0;
  const int32_t lo = off[e], hi = off[e + 1];
  if (lo < 0 || hi < lo || hi > n_total || hi - lo > d.max_arrivals) bad |= ERR_COUNT;
  if (chains(p) && !p->csr_whole) bad |= ERR_COUNT;
  if (!bad) {
    for (const Row& r : rows) {
      if (actions[r.out] < -1 || actions[r.out] >= p->A) bad |= ERR_ACTION;
      if (r.src < 0) continue;    // pending calls are valid by construction
      if (r.q_idx < 0 || (int64_t)r.q_idx >= d.Q) bad |= ERR_QIDX;
      if (r.role < 0) bad |= ERR_ROLE;
      if (r.budget < 1) bad |= ERR_BUDGET;
      if (r.base_svc < 1 || r.base_svc > kSvcMax) bad |= ERR_SVC;
      if (chains(p) && (r.ch.n_steps < 1 || r.ch.n_steps > d.max_steps)) bad |= ERR_STEPS;
    }
  }
  if (bad) { *err |= bad; return; }

  const int32_t t = p->t;
  const int32_t n = (int32_t)rows.size();
  env.arrived += n;
  // S2: admission in id order, tail-drop beyond the queue capacity.
  for (int m = 0; m < d.M; ++m) {
    ModelState& ms = env.models[m];
    const int room = d.qcap - (int)ms.queue.size();
    std::vector<Entry> accepted;
    for (int32_t i = 0; i < n; ++i) {
      const Row& r = rows[i];
      const int32_t a = actions[r.out];
      if (a < 0 || a / d.K != m) continue;
      if ((int)accepted.size() >= room) { ms.rej_overflow += 1; continue; }
      const int32_t depth = a % d.K;
      Entry en;
      en.id = env.next_id + i;
      en.t_arr = t;
      en.svc = r.base_svc * (depth + 1);
      en.budget = r.budget;
      en.key = sort_key(p, t, en.budget, en.svc);
      en.ch = r.ch;
      accepted.push_back(en);
    }
    for (const Entry& en : accepted) { ms.backlog += en.svc; ms.enqueued += 1; }
    // Stable sort of (existing queue ++ newcomers in id order) by key alone:
    // equal keys keep their order, i.e. older ids first.
    ms.queue.insert(ms.queue.end(), accepted.begin(), accepted.end());
    std::stable_sort(ms.queue.begin(), ms.queue.end(),
                     [](const Entry& a, const Entry& b) { return a.key < b.key; });
  }
  for (const Row& r : rows) {
    if (actions[r.out] < 0) env.rej_nomodel += 1;
    else env.hist[actions[r.out]] += 1;
  }
  // S3: per model, fill empty slots s < c_m from the queue head, then advance
  // every busy slot by one tick of service.
  std::vector<Pending> spawned;
  for (int m = 0; m < d.M; ++m) {
    ModelState& ms = env.models[m];
    // forget dispatches that have left every window still to come
    ms.dispatch_ticks.erase(std::remove_if(ms.dispatch_ticks.begin(), ms.dispatch_ticks.end(),
                                           [t](int32_t tau) { return tau <= t - kRpmWindow; }),
                            ms.dispatch_ticks.end());
    int recent = ms.rpm_limit > 0 ? rpm_count(ms, t) : 0;   // dispatches in the window ending at t
    for (int s = 0; s < ms.cap && s < d.max_slots; ++s) {
      Slot& sl = ms.slots[s];
      if (sl.busy || ms.queue.empty()) continue;
      if (ms.rpm_limit > 0 && recent >= ms.rpm_limit) break;   // held back: rate limit reached
      if (ms.rpm_limit > 0) { ms.dispatch_ticks.push_back(t); ++recent; }
      Entry en = ms.queue.front();
      ms.queue.erase(ms.queue.begin());
      sl.busy = true; sl.id = en.id; sl.t_arr = en.t_arr; sl.rem = en.svc; sl.budget = en.budget;
      sl.ch = en.ch;
      ms.backlog -= en.svc;
      ms.started += 1;
      ms.wait_sum += t - en.t_arr;
    }
    for (int s = 0; s < d.max_slots; ++s) {
      Slot& sl = ms.slots[s];
      if (!sl.busy) continue;
      sl.rem -= 1;
      if (sl.rem > 0) continue;
      const int32_t lat = t - sl.t_arr + 1;
      // EWMA with alpha = 1/8 in Q8: ewma += floor((256 lat - ewma) / 8)
      const int64_t delta = (int64_t)lat * 256 - ms.ewma_q8;
      const int64_t step = delta >= 0 ? delta / 8 : -((-delta + 7) / 8);
      ms.ewma_q8 = (int32_t)(ms.ewma_q8 + step);
      ms.completed += 1;
      ms.lat_sum += lat;
      // a call is on time when it completes by its (inherited) deadline
      const bool on_time = lat <= sl.budget;
      ms.slo_met += on_time ? 1 : 0;
      // Sec. 3 cost of the call, latency / beta with beta the query's budget
      // (Eq. 2: the query's cost is the sum over its calls), in Q16
      ms.cost_q16 += ((int64_t)lat << 16) / sl.ch.beta;
      if (chains(p)) {
        if (sl.ch.k + 1 < sl.ch.n_steps) {
          Pending pd;
          pd.ch = sl.ch;
          pd.ch.k += 1;
          pd.deadline = sl.t_arr + sl.budget;   // inherited: the query's deadline
          spawned.push_back(pd);
        } else {
          env.q_done += 1;
          env.q_met += on_time ? 1 : 0;
        }
      }
      sl = Slot();
    }
  }
  env.pending.swap(spawned);
  env.next_id += n;
}

template <class F>
void for_envs(int E, int threads, F f) {
  if (threads <= 1 || E < 2) { for (int e = 0; e < E; ++e) f(e); return; }
  threads = std::min(threads, E);
  std::vector<std::thread> th;
  for (int k = 0; k < threads; ++k)
    th.emplace_back([=, &f] { for (int e = k; e < E; e += threads) f(e); });
  for (auto& x : th) x.join();
}

// Zero state (empty queues and slots, tick 0), the embedding values and the
// per-model logit bias.
void init_state(orc_pool* p, const float* emb, const int32_t* cap, const float* logit_bias) {
  const orc_desc* d = &p->d;
  p->emb.assign(emb, emb + (size_t)d->Q * d->embed_dim);
  p->logit_bias.assign(d->M, 0.0);
  if (logit_bias) for (int m = 0; m < d->M; ++m) p->logit_bias[m] = (double)logit_bias[m];
  p->envs.resize(d->E);
  for (int e = 0; e < d->E; ++e) {
    EnvState& env = p->envs[e];
    env.models.resize(d->M);
    env.hist.assign(p->A, 0);
    for (int m = 0; m < d->M; ++m) {
      env.models[m].slots.resize(d->max_slots);
      env.models[m].cap = cap[e * d->M + m];
    }
  }
}

}  // namespace

extern "C" {

// W[l]: fp32 [widths[l] x in_l] row-major; b[l]: fp32 [widths[l]];
// emb: Q x embed_dim float values; cap: [E*M]; logit_bias: [M] or NULL.
orc_pool* orc_create(const orc_desc* d, const float* const* W, const float* const* b,
                     const float* emb, const int32_t* cap, const float* logit_bias) {
  orc_pool* p = new orc_pool();
  p->d = *d;
  p->d.net = 0;
  p->A = d->M * d->K;
  int in = d->feat_dim;
  for (int l = 0; l < d->n_layers; ++l) {
    const int out = d->widths[l];
    std::vector<double> w((size_t)out * in), bb(out);
    for (size_t i = 0; i < w.size(); ++i)
      w[i] = d->dtype == 1 ? round_bf16((double)W[l][i]) : (double)W[l][i];
    for (int o = 0; o < out; ++o) bb[o] = (double)b[l][o];
    p->W.push_back(w);
    p->b.push_back(bb);
    in = out;
  }
  init_state(p, emb, cap, logit_bias);
  return p;
}

// The dual-pathway executor (Sec. 4.2). P holds, in this order, fp32 arrays:
// W_sem [128 x 2E_d], b_sem, ln_sem gain, ln_sem bias [128]; W_bud [16 x 1],
// b_bud [16]; W_sys [16 x 3M] (input order queue depth | end-to-end latency |
// KV-cache use), b_sys [16]; W_res [64 x 32], b_res, ln_res gain, ln_res bias
// [64]; W_merge [128 x 192], b_merge [128]; W_act [(M K + value_head) x 128],
// b_act. role: fp32 [n_roles x E_d]. d->feat_dim must be E_d + 4M + 1.
orc_pool* orc_create_dual(const orc_desc* d, const float* const* P, const float* role,
                          const float* emb, const int32_t* cap, const float* logit_bias) {
  orc_pool* p = new orc_pool();
  p->d = *d;
  p->d.net = 1;
  p->A = d->M * d->K;
  const int Ed = d->embed_dim, M = d->M, Ao = p->A + d->value_head;
  auto mat = [&](int i, size_t n) {
    std::vector<double> v(n);
    for (size_t k = 0; k < n; ++k) v[k] = d->dtype == 1 ? round_bf16((double)P[i][k]) : (double)P[i][k];
    return v;
  };
  auto vec = [&](int i, size_t n) { return std::vector<double>(P[i], P[i] + n); };
  orc_dual& w = p->dual;
  w.W_sem = mat(0, (size_t)kSem * 2 * Ed); w.b_sem = vec(1, kSem);
  w.g_sem = vec(2, kSem); w.be_sem = vec(3, kSem);
  w.W_bud = mat(4, kBud); w.b_bud = vec(5, kBud);
  w.W_sys = mat(6, (size_t)kSys * 3 * M); w.b_sys = vec(7, kSys);
  w.W_res = mat(8, (size_t)kRes * (kBud + kSys)); w.b_res = vec(9, kRes);
  w.g_res = vec(10, kRes); w.be_res = vec(11, kRes);
  w.W_merge = mat(12, (size_t)kMerge * (kSem + kRes)); w.b_merge = vec(13, kMerge);
  w.W_act = mat(14, (size_t)Ao * kMerge); w.b_act = vec(15, Ao);
  w.role.resize((size_t)d->n_roles * Ed);
  for (size_t k = 0; k < w.role.size(); ++k)
    w.role[k] = d->dtype == 1 ? round_bf16((double)role[k]) : (double)role[k];
  init_state(p, emb, cap, logit_bias);
  return p;
}

// Hidden vectors of one request of env e through the dual-pathway executor:
// out = [h_sem (128) | h_bud (16) | h_sys (16) | h_res (64) | h (128) | logits
// and value (M K + value_head), without the logit bias].
void orc_dual_trace(const orc_pool* p, int e, int32_t q_idx, int32_t role, int32_t budget,
                    double* out) {
  std::vector<double> x;
  features(p, p->envs[e], q_idx, budget, x);
  DualTrace t;
  dual_net(p, x, role, t);
  for (const std::vector<double>* v : {&t.h_sem, &t.h_bud, &t.h_sys, &t.h_res, &t.h, &t.z})
    out = std::copy(v->begin(), v->end(), out);
}

void orc_destroy(orc_pool* p) { delete p; }

int32_t orc_tick(const orc_pool* p) { return p->t; }
int32_t orc_error(const orc_pool* p) { return p->err; }
void orc_clear_error(orc_pool* p) { p->err = 0; }

// Arrival rows of env e the route step reads: single-step pools route
// whatever lies inside the arrays (the schedule step rejects a bad CSR);
// chain pools only a usable CSR entry.
bool route_rows_ok(const orc_pool* p, int e, int32_t n_total, const int32_t* off) {
  if (chains(p)) return csr_ok(p, e, n_total, off);
  return off[e] >= 0 && off[e + 1] <= n_total;
}

// Arrivals: CSR `off` over n_total rows; `n_steps` (chain pools) calls per
// query, NULL for one. Outputs are indexed by row_offsets(): the env's pending
// calls, then its arrivals.
void orc_route(orc_pool* p, int32_t n_total, const int32_t* off, const int32_t* q_idx,
               const int16_t* role, const int16_t* budget, const int16_t* n_steps, double* logits,
               int32_t* actions, int threads) {
  set_csr_whole(p, n_total, off);
  std::vector<int32_t> errs(p->d.E, 0);
  const std::vector<int32_t> ro = row_offsets(p, n_total, off);
  for_envs(p->d.E, threads, [&](int e) {
    std::vector<Row> rows;
    if (route_rows_ok(p, e, n_total, off) || chains(p))
      rows = env_rows(p, e, n_total, off, ro, q_idx, role, budget, nullptr, n_steps);
    route_env(p, e, rows, logits, actions, &errs[e]);
  });
  for (int32_t x : errs) p->err |= x;
}

void orc_schedule(orc_pool* p, int32_t n_total, const int32_t* off, const int32_t* q_idx,
                  const int16_t* role, const int16_t* budget, const int16_t* base_svc,
                  const int16_t* n_steps, const int32_t* actions, int threads) {
  set_csr_whole(p, n_total, off);
  std::vector<int32_t> errs(p->d.E, 0);
  const std::vector<int32_t> ro = row_offsets(p, n_total, off);
  for_envs(p->d.E, threads, [&](int e) {
    std::vector<Row> rows;
    if (csr_ok(p, e, n_total, off) || chains(p))
      rows = env_rows(p, e, n_total, off, ro, q_idx, role, budget, base_svc, n_steps);
    schedule_env(p, e, n_total, off, rows, actions, &errs[e]);
  });
  for (int32_t x : errs) p->err |= x;
  p->t += 1;
}

void orc_route_rl(orc_pool* p, int env_base, int32_t n_total, const int32_t* off,
                  const int32_t* q_idx, const int16_t* role, const int16_t* budget,
                  const int16_t* n_steps, uint32_t seed_lo, uint32_t seed_hi, int greedy,
                  double* logits, int32_t* actions, double* logp, double* entropy, double* value,
                  int threads) {
  set_csr_whole(p, n_total, off);
  std::vector<int32_t> errs(p->d.E, 0);
  const std::vector<int32_t> ro = row_offsets(p, n_total, off);
  for_envs(p->d.E, threads, [&](int e) {
    std::vector<Row> rows;
    if (route_rows_ok(p, e, n_total, off) || chains(p))
      rows = env_rows(p, e, n_total, off, ro, q_idx, role, budget, nullptr, n_steps);
    route_env_rl(p, e, env_base, rows, seed_lo, seed_hi, greedy, logits, actions, logp, entropy,
                 value, &errs[e]);
  });
  for (int32_t x : errs) p->err |= x;
}

// Row offsets of the next route/schedule call (E + 1 entries).
void orc_row_offsets(const orc_pool* p, int32_t n_total, const int32_t* off, int32_t* out) {
  set_csr_whole(p, n_total, off);
  const std::vector<int32_t> ro = row_offsets(p, n_total, off);
  std::copy(ro.begin(), ro.end(), out);
}

// Dual update of the Lagrange multiplier (Eq. 7): over the queries completed
// since the previous update, C_bar = mean of latency / budget (the summed
// floor(2^16 l / beta) of their calls, / 2^16), and
// lambda <- clip(lambda + eta (C_bar - 1), 0, lambda_max). A single-step
// query is one call; a chain's query completes with its last call. No
// completion since the previous update leaves lambda unchanged.
void orc_dual_update(orc_pool* p, double eta, double lambda_max, double* lambda) {
  int64_t n = 0, cost = 0;
  for (const EnvState& env : p->envs) {
    for (const ModelState& ms : env.models) {
      if (!chains(p)) n += ms.completed;
      cost += ms.cost_q16;
    }
    if (chains(p)) n += env.q_done;
  }
  const int64_t dn = n - p->dual_completed, dc = cost - p->dual_cost_q16;
  p->dual_completed = n;
  p->dual_cost_q16 = cost;
  if (dn <= 0) return;
  const double cbar = (double)dc / (65536.0 * (double)dn);
  double l = *lambda + eta * (cbar - 1.0);
  l = l < 0.0 ? 0.0 : (l > lambda_max ? lambda_max : l);
  *lambda = l;
}

void orc_philox4x32_10(const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
  philox4x32_10(ctr, key, out);
}

double orc_gumbel(uint32_t seed_lo, uint32_t seed_hi, int32_t id, int32_t env, int a) {
  return gumbel(seed_lo, seed_hi, id, env, a);
}

// Feature vector of a request of env e as the route step builds it.
void orc_features(const orc_pool* p, int e, int32_t q_idx, int32_t budget, double* out) {
  std::vector<double> x;
  features(p, p->envs[e], q_idx, budget, x);
  std::copy(x.begin(), x.end(), out);
}

double orc_round_bf16(double v) { return round_bf16(v); }
void orc_round_bf16_array(const double* in, double* out, int64_t n) {
  for (int64_t i = 0; i < n; ++i) out[i] = round_bf16(in[i]);
}

void orc_set_enabled(orc_pool* p, int e, int m, int v) { p->envs[e].models[m].enabled = v ? 1 : 0; }
void orc_set_capacity(orc_pool* p, int e, int m, int c) { p->envs[e].models[m].cap = c; }
void orc_set_rpm_limit(orc_pool* p, int e, int m, int r) { p->envs[e].models[m].rpm_limit = r; }

// Blackbox window export: limit, dispatches in the window ending at the last
// completed tick, and the per-tick counts hist[k] of tick (t - 1 - k), k < 60.
void orc_read_rpm(const orc_pool* p, int32_t* limit, int32_t* count, uint8_t* hist) {
  const orc_desc& d = p->d;
  for (int e = 0; e < d.E; ++e)
    for (int m = 0; m < d.M; ++m) {
      const ModelState& ms = p->envs[e].models[m];
      const size_t em = (size_t)e * d.M + m;
      limit[em] = ms.rpm_limit;
      count[em] = rpm_count(ms, p->t - 1);
      for (int k = 0; k < kRpmWindow; ++k) hist[em * kRpmWindow + k] = 0;
      for (int32_t tau : ms.dispatch_ticks) {
        const int k = p->t - 1 - tau;
        if (k >= 0 && k < kRpmWindow) hist[em * kRpmWindow + k] += 1;
      }
    }
}

// State export in the oracle's own layout:
//   env_i32 [E]      next_id
//   env_i64 [E*2]    arrived, rej_nomodel
//   mod_i64 [E*M*14] qlen, busy, ewma_q8, backlog, cap, enabled, rej_overflow,
//                    enqueued, started, completed, slo_met, lat_sum, wait_sum, cost_q16
//   slots   [E*M*max_slots*4] id(-1 if free), t_arr, rem, budget
//   queues  [E*M*qcap*5] key, id, t_arr, svc, budget (zero beyond qlen)
//   hist    [E*A]
void orc_read_state(const orc_pool* p, int32_t* env_i32, int64_t* env_i64, int64_t* mod_i64,
                    int32_t* slots, int32_t* queues, int64_t* hist) {
  const orc_desc& d = p->d;
  for (int e = 0; e < d.E; ++e) {
    const EnvState& env = p->envs[e];
    env_i32[e] = env.next_id;
    env_i64[2 * e] = env.arrived;
    env_i64[2 * e + 1] = env.rej_nomodel;
    for (int a = 0; a < p->A; ++a) hist[(size_t)e * p->A + a] = env.hist[a];
    for (int m = 0; m < d.M; ++m) {
      const ModelState& ms = env.models[m];
      const size_t em = (size_t)e * d.M + m;
      int busy = 0;
      for (const Slot& s : ms.slots) busy += s.busy ? 1 : 0;
      int64_t* o = mod_i64 + em * 14;
      o[0] = (int64_t)ms.queue.size(); o[1] = busy; o[2] = ms.ewma_q8; o[3] = ms.backlog;
      o[4] = ms.cap; o[5] = ms.enabled; o[6] = ms.rej_overflow; o[7] = ms.enqueued;
      o[8] = ms.started; o[9] = ms.completed; o[10] = ms.slo_met; o[11] = ms.lat_sum;
      o[12] = ms.wait_sum; o[13] = ms.cost_q16;
      for (int s = 0; s < d.max_slots; ++s) {
        const Slot& sl = ms.slots[s];
        int32_t* so = slots + (em * d.max_slots + s) * 4;
        so[0] = sl.busy ? sl.id : -1; so[1] = sl.busy ? sl.t_arr : 0;
        so[2] = sl.busy ? sl.rem : 0; so[3] = sl.busy ? sl.budget : 0;
      }
      int32_t* qo = queues + em * (size_t)d.qcap * 5;
      std::memset(qo, 0, sizeof(int32_t) * (size_t)d.qcap * 5);
      for (size_t i = 0; i < ms.queue.size(); ++i) {
        const Entry& en = ms.queue[i];
        qo[i * 5 + 0] = en.key; qo[i * 5 + 1] = en.id; qo[i * 5 + 2] = en.t_arr;
        qo[i * 5 + 3] = en.svc; qo[i * 5 + 4] = en.budget;
      }
    }
  }
}

// Chain state (chain pools): per queued call (queue order) and per slot the
// fields {q_idx, k, n_steps, role0, base, beta}; the pending calls
// {q_idx, k, n_steps, role0, base, beta, deadline} (up to M * max_slots per
// env) with their count; per env the completed and on-time queries.
void orc_read_chain(const orc_pool* p, int32_t* qchain, int32_t* schain, int32_t* pend,
                    int32_t* pcount, int64_t* qcnt) {
  const orc_desc& d = p->d;
  const int PM = d.M * d.max_slots;
  auto put = [](int32_t* o, const Chain& c) {
    o[0] = c.q_idx; o[1] = c.k; o[2] = c.n_steps; o[3] = c.role0; o[4] = c.base; o[5] = c.beta;
  };
  for (int e = 0; e < d.E; ++e) {
    const EnvState& env = p->envs[e];
    for (int m = 0; m < d.M; ++m) {
      const ModelState& ms = env.models[m];
      const size_t em = (size_t)e * d.M + m;
      int32_t* qo = qchain + em * (size_t)d.qcap * 6;
      std::memset(qo, 0, sizeof(int32_t) * (size_t)d.qcap * 6);
      for (size_t i = 0; i < ms.queue.size(); ++i) put(qo + i * 6, ms.queue[i].ch);
      for (int s = 0; s < d.max_slots; ++s) {
        int32_t* so = schain + (em * d.max_slots + s) * 6;
        if (ms.slots[s].busy) put(so, ms.slots[s].ch);
        else std::memset(so, 0, sizeof(int32_t) * 6);
      }
    }
    int32_t* po = pend + (size_t)e * PM * 7;
    std::memset(po, 0, sizeof(int32_t) * (size_t)PM * 7);
    for (size_t i = 0; i < env.pending.size() && (int)i < PM; ++i) {
      put(po + i * 7, env.pending[i].ch);
      po[i * 7 + 6] = env.pending[i].deadline;
    }
    pcount[e] = (int32_t)env.pending.size();
    qcnt[2 * e] = env.q_done;
    qcnt[2 * e + 1] = env.q_met;
  }
}

}  // extern "C"
