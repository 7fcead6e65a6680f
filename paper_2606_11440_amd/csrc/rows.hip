// Rows of a tick in a pool with multi-step agent chains (Sec. 4.3).
//
// An env's rows at tick t are its pending calls (spawned by completions at
// t - 1, in spawn order), then its arrivals in arrival order. The route step
// evaluates the policy on the flat row space; these kernels build it: one
// block scans the per-env row counts into row offsets, then one wave per env
// writes each row's query-embedding row, remaining budget and role.
#include "im_internal.h"
#include "wave.h"

namespace im {
namespace {

constexpr int kScanThreads = 1024;

// Arrivals of env e the route step takes: a CSR entry outside the arrays
// contributes none (the schedule step reports it and skips the env).
__device__ __forceinline__ int32_t usable_arrivals(const RowsArgs& a, int e) {
  const int32_t lo = a.offsets[e], hi = a.offsets[e + 1];
  return (lo < 0 || hi < lo || hi > a.n_total || hi - lo > a.max_arrivals) ? 0 : hi - lo;
}

// One block: exclusive scan of (pending + usable arrivals) over the envs,
// each thread summing a contiguous run of envs.
__global__ __launch_bounds__(kScanThreads) void rows_scan_kernel(RowsArgs a) {
  __shared__ int32_t part[kScanThreads];
  const int tid = threadIdx.x;
  const int32_t t = a.ms[0].t;
  const int32_t* pc = a.pcnt + (size_t)(t & 1) * a.E;
  const int per = (a.E + kScanThreads - 1) / kScanThreads;
  const int e0 = tid * per, e1 = min(e0 + per, a.E);
  int32_t sum = 0;
  for (int e = e0; e < e1; ++e) sum += pc[e] + usable_arrivals(a, e);
  part[tid] = sum;
  __syncthreads();
  // Hillis-Steele inclusive scan of the per-thread sums
  for (int d = 1; d < kScanThreads; d <<= 1) {
    const int32_t v = tid >= d ? part[tid - d] : 0;
    __syncthreads();
    part[tid] += v;
    __syncthreads();
  }
  int32_t run = part[tid] - sum;
  for (int e = e0; e < e1; ++e) {
    a.roff[e] = run;
    run += pc[e] + usable_arrivals(a, e);
  }
  if (tid == kScanThreads - 1) {
    a.roff[a.E] = part[tid];
    a.n_rows[0] = part[tid];
  }
}

// One wave per env: the pending calls' rows (query row, deadline - t, role of
// call k: (role0 + k) mod n_roles), then the arrivals' rows.
__global__ __launch_bounds__(256) void rows_gather_kernel(RowsArgs a) {
  const int lane = threadIdx.x & 63;
  const int e = (int)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (e >= a.E) return;
  const int32_t t = a.ms[0].t;
  const int32_t pc = a.pcnt[(size_t)(t & 1) * a.E + e];
  const int4* pend = a.pend + ((size_t)(t & 1) * a.E + e) * a.pend_cap;
  const int32_t base = a.roff[e];
  for (int i = lane; i < pc; i += 64) {
    const int4 p = pend[i];
    a.rq[base + i] = chain_q(p.x);
    a.rb[base + i] = (int16_t)remaining_budget(p.z, t);
    a.rr[base + i] = (int16_t)(a.n_roles > 0 ? (chain_role0(p.y) + chain_k(p.x)) % a.n_roles : 0);
  }
  const int32_t na = usable_arrivals(a, e);
  const int32_t lo = a.offsets[e];
  for (int i = lane; i < na; i += 64) {
    a.rq[base + pc + i] = a.q_idx[lo + i];
    a.rb[base + pc + i] = a.budget[lo + i];
    a.rr[base + pc + i] = a.role ? a.role[lo + i] : (int16_t)0;
  }
}

}  // namespace

hipError_t launch_rows(const RowsArgs& a, hipStream_t s) {
  hipLaunchKernelGGL(rows_scan_kernel, dim3(1), dim3(kScanThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(rows_gather_kernel, dim3((unsigned)((a.E + 3) / 4)), dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace im
