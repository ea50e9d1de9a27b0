// Varlen tile scheduler.
//
// A packed batch (segments of arbitrary, skewed lengths) is cut into tiles of
// BT tokens per segment.  Under a causal mask the cost of query tile j is
// proportional to j + 1 (it visits tiles 0..j).  The work list comes in two
// orders (plan_lookup in common.hpp): by descending tile level across all
// segments (every workgroup launched early takes one of the longest remaining
// jobs, longest-processing-time-first), or segment by segment, longest
// segment first and each segment's tiles heaviest first (neighbouring
// workgroups then share the rows or keys they stream in L2).  The list is
// never materialised: the plan stores the segments sorted by tile count, the
// first item of every level and the first item of every tile-count group, and
// a kernel maps its item index to (segment, level) with a binary search.  The
// plan costs O(N + max_nt) per launch, also for batches of very many short
// segments.
#pragma once
#include "common.hpp"

namespace pdy {

constexpr int kPlanThreads = 1024;
// tile counts up to this many are binned in LDS (786,432 tokens at 128-token
// tiles); larger ranges bin in the workspace
constexpr int kLdsBuckets = 6144;

// Workspace layout (int32):
//   nt[N] | order[N] | cnt[max_nt] | start[max_nt] | total[1] | before[max_nt]
__host__ __device__ inline size_t plan_ints(int n, int max_nt) {
  return (size_t)2 * n + (size_t)3 * max_nt + 1;
}

// In-place suffix sum over a[0..n) by the whole workgroup: a[j] becomes
// sum_{j' >= j} a[j'] (inclusive) or sum_{j' > j} a[j'] (exclusive).  Each
// thread owns a chunk of consecutive entries counted from the top; the
// threads' totals are scanned within each wave by shuffles and across the
// waves by thread 0 over the wave totals in `wsum` (kPlanThreads / 64 + 1
// entries).  Returns the sum of all entries.
__device__ inline int suffix_sum(int32_t* a, int n, bool inclusive, int32_t* wsum) {
  const int t = threadIdx.x;
  const int lane = t & 63, wv = t >> 6;
  constexpr int kWaves = kPlanThreads / 64;
  const int chunk = (n + kPlanThreads - 1) / kPlanThreads;
  int local = 0;
  for (int c = 0; c < chunk; ++c) {
    const int idx = t * chunk + c;
    if (idx < n) local += a[n - 1 - idx];
  }
  int incl = local;  // inclusive scan of the threads' totals within the wave
  for (int off = 1; off < 64; off <<= 1) {
    const int y = __shfl_up(incl, off, 64);
    if (lane >= off) incl += y;
  }
  if (lane == 63) wsum[wv] = incl;
  __syncthreads();
  if (t == 0) {
    int run = 0;
    for (int w = 0; w < kWaves; ++w) {
      const int v = wsum[w];
      wsum[w] = run;
      run += v;
    }
    wsum[kWaves] = run;
  }
  __syncthreads();
  int run = wsum[wv] + incl - local;  // the totals of all earlier threads
  for (int c = 0; c < chunk; ++c) {
    const int idx = t * chunk + c;
    if (idx < n) {
      const int j = n - 1 - idx;
      const int v = a[j];
      if (inclusive) run += v;
      a[j] = run;
      if (!inclusive) run += v;
    }
  }
  const int total = wsum[kWaves];
  __syncthreads();
  return total;
}

// One schedule to build: segments from cu (cu == nullptr: a single segment
// of single_len tokens, n must be 1), tiles of bt tokens, at most max_nt per
// segment, written to ws.
struct PlanJob {
  const int32_t* cu;
  int n;
  int bt;
  int max_nt;
  int single_len;
  int32_t* ws;
};
// Up to two schedules per launch (the backward needs one over key tiles and
// one over query tiles): workgroup b builds job[b].
struct PlanJobs {
  PlanJob job[2];
};

__device__ inline void build_plan(const int32_t* __restrict__ cu, int n, int bt, int max_nt,
                                  int single_len, int32_t* __restrict__ ws) {
  int32_t* nt = ws;
  int32_t* order = nt + n;
  int32_t* cnt = order + n;
  int32_t* start = cnt + max_nt;
  int32_t* total = start + max_nt;
  int32_t* before = total + 1;
  const int t = threadIdx.x;
  __shared__ int32_t wsum[kPlanThreads / 64 + 1];
  // per-count histogram and placement cursors: in LDS when they fit (many
  // segments with the same count then contend in LDS, not in L2)
  __shared__ int32_t lds_hist[kLdsBuckets];
  __shared__ int32_t lds_cur[kLdsBuckets];
  const bool in_lds = max_nt <= kLdsBuckets;
  int32_t* hist = in_lds ? lds_hist : cnt;
  int32_t* cur = in_lds ? lds_cur : start;

  // 1. tiles per segment, and hist[v - 1] = number of segments with v tiles
  for (int j = t; j < max_nt; j += kPlanThreads) {
    hist[j] = 0;
    cur[j] = 0;
  }
  __syncthreads();
  for (int s = t; s < n; s += kPlanThreads) {
    const int len = cu ? cu[s + 1] - cu[s] : single_len;
    int v = (len + bt - 1) / bt;
    v = v < max_nt ? v : max_nt;  // max_seqlen is a caller-guaranteed bound
    nt[s] = v;
    if (v > 0) atomicAdd(&hist[v - 1], 1);
  }
  __syncthreads();

  // 2. cnt[j] = number of segments with more than j tiles
  if (in_lds) {
    for (int j = t; j < max_nt; j += kPlanThreads) cnt[j] = hist[j];
    __syncthreads();
  }
  suffix_sum(cnt, max_nt, true, wsum);

  // 3. order: segments by tile count, most first (a counting sort: the ones
  // with v tiles fill positions [cnt[v], cnt[v - 1]) through the per-count
  // cursor).  The order among segments with the same count depends on the
  // atomics' timing, which changes which workgroup runs an item but not what
  // the item computes.
  for (int s = t; s < n; s += kPlanThreads) {
    const int v = nt[s];
    if (v > 0) order[(v < max_nt ? cnt[v] : 0) + atomicAdd(&cur[v - 1], 1)] = s;
  }
  __syncthreads();

  // 4. start[j] = sum_{j' > j} cnt[j'] (first item of level j); total items;
  // before[j] = tiles of the segments with more than j + 1 tiles (in the
  // segment-major order the segments with exactly j + 1 tiles start there)
  for (int j = t; j < max_nt; j += kPlanThreads) {
    start[j] = cnt[j];
    before[j] = (j + 1) * (cnt[j] - (j + 1 < max_nt ? cnt[j + 1] : 0));
  }
  __syncthreads();
  const int items = suffix_sum(start, max_nt, false, wsum);
  suffix_sum(before, max_nt, false, wsum);
  if (t == 0) *total = items;
}

__global__ void __launch_bounds__(kPlanThreads) plan_kernel(PlanJobs jobs) {
  const PlanJob& j = jobs.job[blockIdx.x];
  build_plan(j.cu, j.n, j.bt, j.max_nt, j.single_len, j.ws);
}

}  // namespace pdy
