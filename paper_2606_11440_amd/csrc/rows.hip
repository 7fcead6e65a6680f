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

// One block: exclusive scan of (pending + usable arrivals) over the envs.
// Each thread holds the counts of kPer consecutive envs in registers; wave
// scans by shuffles, the 16 wave totals scanned by the first wave; blocks of
// 1024 * kPer envs in sequence with a carried total.
constexpr int kPer = 8;

__device__ __forceinline__ int32_t wave_incl_scan(int32_t x, int lane) {
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int32_t y = __shfl_up(x, d, 64);
    if (lane >= d) x += y;
  }
  return x;
}

__global__ __launch_bounds__(kScanThreads) void rows_scan_kernel(RowsArgs a) {
  constexpr int NWAVE = kScanThreads / 64;
  __shared__ int32_t wsum[NWAVE];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int32_t t = a.ms[0].t;
  const int32_t* pc = a.pcnt + (size_t)(t & 1) * a.E;
  // The rows are laid out by a scan over the arrival CSR, so it must be one
  // monotone partition of [0, n_total); otherwise no arrival is usable (every
  // env then skips the tick in the schedule step).
  int broken = 0;
  if (tid == 0) broken = a.offsets[0] != 0 || a.offsets[a.E] != a.n_total;
  for (int e = tid; e < a.E; e += kScanThreads) broken |= a.offsets[e + 1] < a.offsets[e];
  const bool whole = __syncthreads_or(broken) == 0;
  int32_t carry = 0;
  for (int base = 0; base < a.E; base += kScanThreads * kPer) {
    int32_t c[kPer];
    int32_t sum = 0;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int e = base + tid * kPer + j;
      c[j] = e < a.E ? pc[e] + (whole ? usable_arrivals(a, e) : 0) : 0;
      sum += c[j];
    }
    const int32_t x = wave_incl_scan(sum, lane);
    if (lane == 63) wsum[w] = x;
    __syncthreads();
    if (w == 0) {
      const int32_t v = wave_incl_scan(lane < NWAVE ? wsum[lane] : 0, lane);
      if (lane < NWAVE) wsum[lane] = v;
    }
    __syncthreads();
    int32_t run = carry + (w > 0 ? wsum[w - 1] : 0) + x - sum;
#pragma unroll
    for (int j = 0; j < kPer; ++j) {
      const int e = base + tid * kPer + j;
      if (e < a.E) a.roff[e] = run;
      run += c[j];
    }
    carry += wsum[NWAVE - 1];
    __syncthreads();   // wsum is rewritten by the next block of envs
  }
  if (tid == 0) {
    a.roff[a.E] = carry;
    a.n_rows[0] = carry;
    a.n_rows[1] = whole ? 0 : 1;
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
  const int32_t na = a.n_rows[1] == 0 ? usable_arrivals(a, e) : 0;   // written by the scan kernel
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
