/* inframind.h -- C ABI of the batched route-and-schedule tick on MI355X.
 *
 * A pool holds E independent simulated serving pools ("envs"), each with M
 * models (LLM services) that own a request queue and c_m service slots.
 * Every tick, for every env, in parallel on the GPU:
 *   route    -- each arriving request (one agent step) gets a feature vector
 *               from its query embedding, its budget and the env's live load
 *               (Sec. 3 "State", Eq. 1: query embedding, remaining budget,
 *               per-model queue depth, end-to-end latency, KV-cache use), a
 *               policy MLP scores all M*K joint actions and a masked argmax
 *               picks one (Sec. 3 "Action": model = a / K, depth = a % K;
 *               Sec. 4.2 executor, deployed greedily);
 *   schedule -- routed requests are admitted to their model's queue, which is
 *               kept ordered by an integer key (Sec. 4.3: deadline
 *               t_arrive + budget, earliest first; here by default the latest
 *               start time = deadline - service time, ties by request id);
 *               each model fills its free service slots from the queue head,
 *               advances service by one tick and records completions (bounded
 *               concurrency as vLLM's max_num_seqs, Table 5; latency signal
 *               an exponential moving average, Sec. 5.4).
 *
 * Conventions for every call:
 *   - Pointers marked "device" are device memory of the pool's GPU; "host"
 *     pointers are ordinary host memory. Caller-owned buffers must stay valid
 *     until the stream work that uses them has finished.
 *   - `stream` is a hipStream_t (NULL = the default stream). All tick calls
 *     are stream-ordered and asynchronous; only im_read_state, im_write_state,
 *     im_get_error and im_pool_create/im_destroy synchronise.
 *   - Invalid arguments return IM_EINVAL synchronously and change nothing.
 *     Data-dependent errors found on the device (see IM_ERR_*) set a sticky
 *     error word and leave the offending env's state untouched for that tick;
 *     they are reported by im_get_error.
 *   - A pool is not thread-safe; distinct pools are independent.
 */
#ifndef INFRAMIND_H
#define INFRAMIND_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  IM_OK = 0,
  IM_EINVAL = -1,      /* bad argument (nothing changed)                 */
  IM_ENOMEM = -2,      /* device allocation failed                       */
  IM_EHIP = -3,        /* a HIP runtime call or kernel launch failed     */
  IM_EDEVICE = -4,     /* sticky device error word is non-zero           */
  IM_ESTATE = -5,      /* im_write_state given an inconsistent snapshot  */
  IM_EUNSUPPORTED = -6 /* valid description with no kernel for its shape */
} im_status;

typedef enum { IM_F32 = 0, IM_BF16 = 1 } im_dtype;

/* Queue order (Sec. 4.3). SLACK: key = t_arrive + budget - svc (latest start
 * time; ordering by it orders by slack at every tick). DEADLINE: key =
 * t_arrive + budget (the paper's EDF). FCFS: key = t_arrive (the baseline of
 * the Table 3 ablation). Ties are broken by request id in every mode. */
typedef enum { IM_KEY_SLACK = 0, IM_KEY_DEADLINE = 1, IM_KEY_FCFS = 2 } im_key_mode;

/* Bits of the sticky device error word. */
#define IM_ERR_QIDX   1   /* q_idx outside [0, n_queries)                          */
#define IM_ERR_COUNT  2   /* offsets not a CSR of n_total rows, or n_e > max; in a
                           * chain pool an offsets array that is not one monotone
                           * partition of [0, n_total) skips every env            */
#define IM_ERR_BUDGET 4   /* budget < 1                                            */
#define IM_ERR_SVC    8   /* base_svc outside [1, IM_SVC_MAX]                      */
#define IM_ERR_ACTION 16  /* action outside [-1, M*K)                              */
#define IM_ERR_ROLE   32  /* role outside [0, n_roles) (dual-pathway pools)          */
#define IM_ERR_STEPS  64  /* n_steps outside [1, max_steps] (chain pools)          */

/* Limits of this build. */
#define IM_SVC_MAX     4095   /* largest base service time (ticks)              */
#define IM_MAX_MODELS  32
#define IM_MAX_DEPTHS  16
#define IM_MAX_ACTIONS 64     /* M*K                                            */
#define IM_MAX_SLOTS   8
#define IM_MAX_QCAP    16384
#define IM_MAX_FEAT    512
#define IM_MAX_ROLES   4096
#define IM_MAX_STEPS   15     /* calls per query of a chain pool                */

/* Policy network of a pool (Sec. 4.2). MLP: a plain MLP over the feature
 * vector (widths from the description). DUAL: the paper's dual-pathway
 * executor with its fixed widths (see im_dual_net). */
typedef enum { IM_NET_MLP = 0, IM_NET_DUAL = 1 } im_net;

/* Pool description.
 *   n_envs        E >= 1 independent envs
 *   n_models      M in [1, IM_MAX_MODELS]; n_depths K in [1, IM_MAX_DEPTHS]; M*K <= 64
 *   queue_cap     per-(env, model) queue capacity in [1, IM_MAX_QCAP]
 *   max_slots     slots per model in [1, IM_MAX_SLOTS]; capacities lie in [0, max_slots]
 *   embed_dim     E_d, query-embedding width (>= 1)
 *   feat_dim      D_in >= E_d + 4M + 1, <= IM_MAX_FEAT. Feature layout:
 *                 [embedding (E_d) | queue depth of every model (M) | busy/c_m (M) |
 *                  latency EWMA/(256 B) (M) | backlog/(c_m B) (M) | budget/B | 0...]
 *                 with B = budget_max and every reciprocal rounded once to fp32.
 *   n_layers      2 or 3; widths[0..n_layers-1] are the layer output widths,
 *                 hidden widths equal, in {32, 64, 128, 256, 512} (512 bf16 only),
 *                 widths[n_layers-1] == M*K + value_head
 *   dtype         IM_F32: fp32 weights and activations; IM_BF16: bf16 weights,
 *                 inputs and hidden activations (round to nearest even), fp32
 *                 accumulation, biases and logits
 *   key_mode      im_key_mode
 *   max_arrivals_per_env_tick  largest n_e accepted (>= 1)
 *   budget_max    B >= 1, normaliser of the budget and latency features
 *   value_head    0 or 1. With 1 the last layer has one more row, row M*K,
 *                 whose output is the state value V(s) = w_val . h + b_val of
 *                 the last hidden layer h (Sec. 4.2 "Decision"); it gets no
 *                 logit bias and takes no part in routing.
 *   net           im_net; IM_NET_DUAL pools are created by im_pool_create_dual,
 *                 which ignores feat_dim, n_layers and widths
 *   n_roles       IM_NET_DUAL: rows of the role-embedding table, in
 *                 [1, IM_MAX_ROLES]; ignored for IM_NET_MLP
 *   max_steps     0 or 1: every request is a single call. 2..IM_MAX_STEPS: a
 *                 chain pool (multi-step agent chains, Sec. 4.3): an arriving
 *                 query is a sequence of n_steps <= max_steps calls run one
 *                 after the other; when call k completes at tick t, call k + 1
 *                 is routed at tick t + 1 with the query's deadline
 *                 t_arrive + budget, i.e. with the remaining budget
 *                 deadline - (t + 1) (which may be <= 0). Every call of a
 *                 query has the query's embedding row and base service time;
 *                 in dual-pathway pools call k has role (role + k) mod n_roles.
 *                 Chain pools need n_queries <= 2^24 and, for IM_NET_DUAL,
 *                 n_roles <= 32. */
typedef struct {
  int32_t n_envs, n_models, n_depths, queue_cap, max_slots;
  int32_t embed_dim, feat_dim, n_layers;
  int32_t widths[4];
  int32_t dtype, key_mode, max_arrivals_per_env_tick, budget_max;
  int32_t value_head;
  int32_t net, n_roles;
  int32_t max_steps;
} im_pool_desc;

/* The arrivals of ONE tick, in env-major CSR order (all device memory).
 *   offsets  [E+1]  rows of env e are [offsets[e], offsets[e+1]); offsets[0] = 0,
 *                   offsets[E] = n_total
 *   q_idx    [n]    row of the query-embedding table
 *   budget   [n]    time budget in ticks (>= 1)
 *   base_svc [n]    service time at depth 0 in ticks; at depth d it is base_svc*(d+1)
 *   role     [n]    row of the role-embedding table: the role of the agent
 *                   step that issues the request (Sec. 4.2). Required by
 *                   IM_NET_DUAL pools, ignored (may be NULL) by IM_NET_MLP pools
 *   n_steps  [n]    chain pools: calls of the arriving query, in [1, max_steps]
 *                   (required); ignored (may be NULL) by single-call pools
 * Within an env, rows are in arrival order; request ids are assigned in that
 * order, continuing from the env's next_id.
 *
 * Rows of a tick. In single-call pools the rows are the arrivals and every
 * per-row output is indexed like them. In chain pools an env's rows are its
 * pending calls (in the order they were spawned: by model, then slot), then
 * its arrivals; per-row outputs are indexed by the row offsets im_get_rows
 * reports (env e: rows [offsets[e], offsets[e+1])), and caller buffers must
 * hold n_total + n_envs * n_models * max_slots rows. Request ids follow the
 * row order. */
typedef struct {
  const int32_t* offsets;
  const int32_t* q_idx;
  const int16_t* budget;
  const int16_t* base_svc;
  const int16_t* role;
  const int16_t* n_steps;
  int32_t n_total;
} im_arrivals;

typedef struct im_pool im_pool;

/* Create a pool (Sec. 4.2 policy weights, Sec. 4.3 queues, all state zero:
 * empty queues and slots, tick 0, next_id 0, enabled = 1).
 *   W[l]        host fp32 [widths[l] x in_l] row-major (in_0 = feat_dim);
 *               copied (and rounded to bf16 for IM_BF16) into the pool
 *   b[l]        host fp32 [widths[l]]; copied
 *   emb         device [n_queries x embed_dim], fp32 (IM_F32) or bf16 bits
 *               (IM_BF16), row-major; BORROWED: must outlive the pool
 *   capacity    host int32 [E*M], c_m per (env, model) in [0, max_slots]
 *   logit_bias  host fp32 [M] added to the logits of model m's actions, or NULL
 * Returns IM_EINVAL / IM_EUNSUPPORTED / IM_ENOMEM / IM_EHIP on failure
 * (*out untouched). Synchronises `stream`. */
im_status im_pool_create(const im_pool_desc* desc, const float* const* W, const float* const* b,
                         const void* emb, int64_t n_queries, const int32_t* capacity,
                         const float* logit_bias, void* stream, im_pool** out);

/* Parameters of the paper's dual-pathway executor (Sec. 4.2), all host fp32,
 * matrices [out x in] row-major, copied at creation (matrices and role table
 * rounded to bf16, biases and LayerNorm parameters kept in fp32):
 *   semantic pathway  h_sem = LN(ReLU(W_sem [e_q | e_r] + b_sem)), 128 wide;
 *                     W_sem [128 x 2 E_d], b_sem, ln_sem_gain, ln_sem_bias [128]
 *   budget head       h_bud = ReLU(W_bud b + b_bud), 16 wide; W_bud [16 x 1], b_bud [16],
 *                     b = budget / budget_max (the normalised remaining budget)
 *   system head       h_sys = ReLU(W_sys [d_queue | d_e2e | d_kv] + b_sys), 16 wide;
 *                     W_sys [16 x 3M], b_sys [16]; per model the queue-depth,
 *                     latency-EWMA and busy-slot features of the MLP feature
 *                     vector (im_pool_desc) in that order
 *   resource pathway  h_res = LN(ReLU(W_res [h_bud | h_sys] + b_res)), 64 wide;
 *                     W_res [64 x 32], b_res, ln_res_gain, ln_res_bias [64]
 *   decision          h = ReLU(W_merge [h_sem | h_res] + b_merge), 128 wide;
 *                     W_merge [128 x 192], b_merge [128]; logits W_act h + b_act,
 *                     W_act [(M*K + value_head) x 128], b_act [M*K + value_head]
 *                     (row M*K: the value head V(s))
 *   role_emb          [n_roles x E_d] role-embedding table e_r
 * LayerNorm: (x - mean) / sqrt(var + 1e-5) * gain + bias over the vector, with
 * the biased variance. Every vector entering a matrix product is bf16. */
typedef struct {
  const float *W_sem, *b_sem, *ln_sem_gain, *ln_sem_bias;
  const float *W_bud, *b_bud;
  const float *W_sys, *b_sys;
  const float *W_res, *b_res, *ln_res_gain, *ln_res_bias;
  const float *W_merge, *b_merge;
  const float *W_act, *b_act;
  const float *role_emb;
} im_dual_net;

/* Create a pool whose policy is the dual-pathway executor (desc->net must be
 * IM_NET_DUAL, desc->dtype IM_BF16; embed_dim in {64, 128, 256, 384}; M*K +
 * value_head <= 32). The query-embedding table, capacities, logit bias,
 * stream and errors are as for im_pool_create; every other call works on the
 * pool unchanged, with arrivals carrying a role per row. */
im_status im_pool_create_dual(const im_pool_desc* desc, const im_dual_net* net, const void* emb,
                              int64_t n_queries, const int32_t* capacity, const float* logit_bias,
                              void* stream, im_pool** out);

/* Route one tick (Sec. 3 Eq. 1 features, Sec. 4.2 policy, masked argmax).
 * Reads the state left by the previous tick; does not change the state.
 *   actions  device int32 [n_total] out: chosen joint action, -1 when no
 *            action is valid (model disabled, c_m = 0 or its queue full) or
 *            the row's q_idx is out of range (IM_ERR_QIDX is raised) or, in
 *            a dual-pathway pool, its role (IM_ERR_ROLE)
 *   logits   device fp32 [n_total x M*K] out (post logit-bias, pre-mask), or NULL
 * Argmax ties go to the lowest action index. */
im_status im_route(im_pool* pool, const im_arrivals* arr, int32_t* actions, float* logits,
                   void* stream);

/* Outputs of im_route_sample (device memory, caller-owned; one entry per
 * arrival row). Any pointer but `actions` may be NULL to skip that output. */
typedef struct {
  int32_t* actions;   /* int32 [n_total]: chosen joint action, -1 as in im_route          */
  float* logp;        /* fp32 [n_total]: log pi(action | s); 0 when the action is -1      */
  float* entropy;     /* fp32 [n_total]: entropy of pi(. | s); 0 when no action is valid  */
  float* value;       /* fp32 [n_total]: V(s) (pools with value_head = 1 only)            */
  float* logits;      /* fp32 [n_total x M*K]: as in im_route                             */
} im_policy_out;

/* Route one tick for an RL rollout (Sec. 4.4: the executor's PPO objective,
 * Eq. 5, needs the action's log-probability, the policy entropy and the state
 * value). pi(a | s) is the softmax of the logits over the valid actions
 * (masked as in im_route). With greedy = 0 the action is drawn from pi by the
 * Gumbel-max trick: argmax over valid a of z_a + G_a with
 * G_a = -ln(-ln U_a), U_a = (top 23 bits of word a % 4 of the Philox4x32-10
 * block (Salmon et al., SC 2011) with counter (request id, env, a / 4, 0) and
 * key (seed low 32 bits, seed high 32 bits)) + 1/2, times 2^-23. Request ids
 * are the per-env ids im_schedule assigns (next_id + position in the env's
 * rows), so every request gets its own noise for a given seed. With
 * greedy = 1 the action is the masked argmax of im_route. Reads the state,
 * does not change it. IM_EINVAL if value is requested from a pool without a
 * value head. */
im_status im_route_sample(im_pool* pool, const im_arrivals* arr, uint64_t seed, int32_t greedy,
                          const im_policy_out* out, void* stream);

/* Rows of the current tick of a chain pool (device pointers owned by the
 * pool). They are rebuilt from the pending calls and the arrivals by every
 * im_route, im_route_sample, im_schedule and im_tick call (before it routes or
 * schedules) and stay valid until the next such call.
 *   offsets  [n_envs + 1] row range of each env (pending calls first)
 *   n_rows   [2] rows of the tick, then 1 when the arrival offsets are not one
 *            monotone partition of [0, n_total): no arrival is then routed and
 *            every env skips the tick with IM_ERR_COUNT
 *   q_idx, budget, role  per row: query-embedding row, budget the call is
 *            routed with (the remaining budget for a pending call), role
 * IM_EINVAL for a single-call pool. */
typedef struct {
  const int32_t* offsets;
  const int32_t* n_rows;
  const int32_t* q_idx;
  const int16_t* budget;
  const int16_t* role;
} im_rows;
im_status im_get_rows(im_pool* pool, im_rows* out);

/* Schedule one tick with the given actions (any actions in [-1, M*K), e.g.
 * sampled ones): admission in id order with tail-drop beyond queue_cap, keys
 * per key_mode, service of every model, accounting; then the tick advances.
 * The scheduler of Sec. 4.3 (each model's queue served earliest deadline
 * first; chain pools: a call inherits its query's deadline), the bounded
 * per-model concurrency of Table 5 (c_m slots) and the latency moving
 * average of Sec. 5.4. The load statistics the next im_route reads (Sec. 3,
 * Eq. 1) are refreshed here.
 *   actions  device int32 [n_total] (chain pools: the rows of im_get_rows) */
im_status im_schedule(im_pool* pool, const im_arrivals* arr, const int32_t* actions, void* stream);

/* im_route followed by im_schedule with the actions it chose: one step of
 * the executor's decision (Sec. 4.2, masked argmax over the joint actions of
 * Sec. 3) and of the scheduler (Sec. 4.3) for every env.
 *   actions_out  device int32 [n_total] receiving the actions, or NULL
 *                (then a pool-owned buffer is used) */
im_status im_tick(im_pool* pool, const im_arrivals* arr, int32_t* actions_out, void* stream);

/* im_tick for callers that cannot allocate device memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * actions passed from the route step to the schedule step are staged in a
 * static device array of 2^21 rows (8 MiB; each GPU holds its own from the
 * first pool created on it until the process ends) instead of a pool buffer.
 * Allocates nothing. All calls on one GPU share that array: calls that
 * overlap on one GPU (concurrent streams, other threads) race and must not be
 * issued. IM_EINVAL when the tick's rows (n_total, plus n_envs * n_models *
 * max_slots pending calls in a chain pool) exceed 2^21; the results equal
 * im_tick's. */
im_status im_tick_noalloc(im_pool* pool, const im_arrivals* arr, void* stream);

/* Free every resource of the pool (synchronises). NULL is ignored. */
void im_destroy(im_pool* pool);

/* ---- state snapshot (host memory; synchronises) -------------------------- */

typedef struct {            /* a queued request, in service order             */
  int32_t key, id, t_arr;   /* sort key, per-env request id, arrival tick     */
  uint16_t svc;             /* service time (ticks)                           */
  int16_t budget;           /* budget (ticks; a chain's later call: what is left, may be <= 0) */
} im_entry;

typedef struct {            /* a service slot; id = -1 when free              */
  int32_t id, t_arr, rem, budget;
} im_slot;

typedef struct {
  int32_t qlen, busy, ewma_q8, backlog, capacity, enabled, _pad0, _pad1;
  int64_t rej_overflow, enqueued, started, completed, slo_met, lat_sum, wait_sum;
  int64_t cost_q16;         /* sum over completions of floor(2^16 latency / budget) */
  int32_t rpm_limit;        /* blackbox rate limit per 60 ticks (0: not rate-limited)   */
  int32_t rpm_count;        /* dispatches in the 60 ticks up to the last completed tick */
  uint8_t rpm_hist[60];     /* rpm_hist[k]: dispatches at tick (tick - 1 - k)           */
  int32_t _pad2;
} im_model_state;

typedef struct {
  int64_t arrived, rej_nomodel;   /* rows (calls) seen; rows routed to no model   */
  int32_t next_id, _pad;
  int64_t q_done, q_met;          /* chain pools: queries whose last call completed;
                                     of them, those completed by their deadline */
} im_env_state;

/* Copy the state of envs [env_begin, env_begin + env_count) to host memory:
 * what the executor observes (Sec. 3, Eq. 1: per-model queue depth, latency
 * moving average, busy slots standing in for KV-cache use), every queue in
 * the scheduler's service order (Sec. 4.3) and the accounting counters.
 *   tick    out: ticks completed so far
 *   envs    [count], models [count*M], slots [count*M*max_slots],
 *   queues  [count*M*queue_cap] (entries beyond qlen are zeroed),
 *   hist    [count*M*K] routed requests per action
 * Any output pointer may be NULL to skip it. */
im_status im_read_state(im_pool* pool, int32_t env_begin, int32_t env_count, int32_t* tick,
                        im_env_state* envs, im_model_state* models, im_slot* slots,
                        im_entry* queues, int64_t* hist);

/* The chain words of a call (chain pools): its query's embedding row, its
 * index k among the query's n_steps calls, the role of the query's first
 * call, the base service time and the query's budget. */
typedef struct {
  int32_t q_idx;
  int16_t k, n_steps, role0, base_svc;
  int32_t beta;
} im_chain;

typedef struct {            /* a call waiting for the next tick's route step   */
  im_chain ch;
  int32_t deadline;         /* the query's deadline t_arrive + beta           */
} im_pending;

/* Chain state of envs [env_begin, env_begin + env_count) (chain pools; host
 * memory; synchronises): the chain words of every queued call, in the order
 * of im_read_state's queues ([count*M*queue_cap]), and of every busy slot
 * ([count*M*max_slots], zero for a free slot); the pending calls of each env
 * ([count*M*max_slots]) and their number ([count]). Any pointer may be NULL.
 * IM_EINVAL for a single-call pool. */
im_status im_read_chain_state(im_pool* pool, int32_t env_begin, int32_t env_count, im_chain* queues,
                              im_chain* slots, im_pending* pending, int32_t* pending_count);

/* Overwrite the state of envs [env_begin, env_begin + env_count) and the tick
 * from host memory (same layout as im_read_state; all pointers required).
 * Returns IM_ESTATE without changing anything if the snapshot is
 * inconsistent: a queue not strictly increasing in (key, id); qlen, busy or
 * backlog not matching the queues and slots; a queued key other than the key
 * mode's function of its arrival tick, budget and service time; an arrival
 * tick outside [0, tick), an id at or above the env's next id, a service time
 * outside [1, IM_SVC_MAX * n_depths], a budget below 1; other bounds.
 * IM_EUNSUPPORTED for chain pools (restored with im_write_chain_state). */
im_status im_write_state(im_pool* pool, int32_t env_begin, int32_t env_count, int32_t tick,
                         const im_env_state* envs, const im_model_state* models,
                         const im_slot* slots, const im_entry* queues, const int64_t* hist);

/* Restore a chain pool (checkpoint/resume of the multi-step chains of
 * Sec. 4.3, whose calls inherit their query's deadline): the snapshot of
 * im_write_state (queued and running calls may carry a budget <= 0: what is
 * left of their query's) plus, in the layouts of im_read_chain_state, the
 * chain words of every queued call (queue order) and of every busy slot, and
 * each env's pending calls ([count*M*max_slots], pending_count [count]),
 * which the next im_route routes first. All pointers required (host memory;
 * synchronises). IM_ESTATE without any change if inconsistent (the checks of
 * im_write_state; chain words out of range: q_idx outside [0, n_queries),
 * k outside [0, n_steps), n_steps outside [1, max_steps], base_svc outside
 * [1, IM_SVC_MAX] or not dividing the queued service time in at most
 * n_depths steps, beta outside [1, 32767], role0 outside [0, n_roles); a
 * pending call with k = 0 or a count above M*max_slots). IM_EINVAL for a
 * single-call pool. */
im_status im_write_chain_state(im_pool* pool, int32_t env_begin, int32_t env_count, int32_t tick,
                               const im_env_state* envs, const im_model_state* models,
                               const im_slot* slots, const im_entry* queues, const int64_t* hist,
                               const im_chain* queue_chains, const im_chain* slot_chains,
                               const im_pending* pending, const int32_t* pending_count);

/* Dual update of the Lagrange multiplier (Sec. 4.4, Eq. 7; App. C with no
 * monetary budget): over the requests completed since the previous call (or
 * since pool creation), C_bar = mean of latency / budget (each term
 * floor(2^16 latency / budget) / 2^16, the cost of Eq. 2), then
 * lambda <- clip(lambda + eta (C_bar - 1), 0, lambda_max) in fp64. With no
 * completion in between, lambda is unchanged.
 *   lambda  device fp64 [1], in/out
 * Stream-ordered; IM_EINVAL for eta < 0 or lambda_max < 0. */
im_status im_dual_update(im_pool* pool, double eta, double lambda_max, double* lambda, void* stream);

/* Launch shapes, for operations and tests of determinism (calls made after
 * it use the new shapes; no result depends on them; not stream-ordered):
 *   route_blocks  grid of the persistent route kernels: -1 one block per
 *                 compute unit (the default), n > 0 at most n blocks sharing
 *                 the tick's row tiles, 0 the kernels that launch one wave
 *                 per row tile instead
 *   sched_waves   envs (one wave each) per workgroup of the schedule step:
 *                 1, 2 or 4 (the default); 0 keeps the current value
 * IM_EINVAL for other values. */
im_status im_set_launch(im_pool* pool, int32_t route_blocks, int32_t sched_waves);

/* Host knobs (stream-ordered): take a model out of routing, or change its
 * number of service slots (requests in slots >= the new capacity finish but
 * are not replaced), or make it a blackbox (API) model with a rate limit
 * (Sec. 5.5, App. C): with rpm_limit > 0 a queued request enters a free slot
 * only while fewer than rpm_limit requests entered its slots in the last 60
 * ticks (the rest wait in its queue), and its queue-depth feature becomes
 * (requests dispatched in the last 60 ticks) * fp32(1 / rpm_limit) instead of
 * queue length / queue_cap. 0 restores the white-box model; dispatches stop
 * being recorded and the window empties as they age out. rpm_limit in
 * [0, 2^30]. The first limit > 0 set on a pool switches its schedule step to
 * the variant that tracks the windows; schedule calls captured into a graph
 * before that keep the variant they were captured with. */
im_status im_set_enabled(im_pool* pool, int32_t env, int32_t model, int32_t enabled, void* stream);
im_status im_set_capacity(im_pool* pool, int32_t env, int32_t model, int32_t capacity,
                          void* stream);
im_status im_set_rpm_limit(im_pool* pool, int32_t env, int32_t model, int32_t rpm_limit,
                           void* stream);

/* Sticky device error word (IM_ERR_* bits). Synchronises. Returns IM_EDEVICE
 * when non-zero. im_clear_error zeroes it. */
im_status im_get_error(im_pool* pool, int32_t* bits);
im_status im_clear_error(im_pool* pool);

/* Description of the last failing call on this pool (or of the last failed
 * im_pool_create when pool is NULL). Never NULL. */
const char* im_last_error(const im_pool* pool);

#ifdef __cplusplus
}
#endif
#endif /* INFRAMIND_H */
