// Varlen tile scheduler.
//
// A packed batch (segments of arbitrary, skewed lengths) is cut into tiles of
// BT tokens per segment.  Under a causal mask the cost of query tile j is
// proportional to j + 1 (it visits tiles 0..j), so the work list is ordered by
// descending tile level across all segments: every workgroup launched early
// takes one of the longest remaining jobs (longest-processing-time-first),
// which balances the tail of a launch when lengths are skewed.  The list is
// never materialised: the plan stores the segments sorted by tile count and
// the first item index of every level, and a kernel maps its item index to
// (segment, level) with a binary search (plan_lookup in common.hpp).
#pragma once
#include "common.hpp"

namespace pdy {

constexpr int kPlanThreads = 1024;

// Workspace layout (int32): nt[N] | order[N] | cnt[max_nt] | start[max_nt] | total[1]
__host__ __device__ inline size_t plan_ints(int n, int max_nt) {
  return (size_t)2 * n + (size_t)2 * max_nt + 1;
}

// cu == nullptr: a single segment of single_len tokens (n must be 1)
__global__ void __launch_bounds__(kPlanThreads)
plan_kernel(const int32_t* __restrict__ cu, int n, int bt, int max_nt, int single_len,
            int32_t* __restrict__ ws) {
  int32_t* nt = ws;
  int32_t* order = nt + n;
  int32_t* cnt = order + n;
  int32_t* start = cnt + max_nt;
  int32_t* total = start + max_nt;
  const int t = threadIdx.x;
  __shared__ int32_t part[kPlanThreads];

  // 1. tiles per segment
  for (int s = t; s < n; s += kPlanThreads) {
    const int len = cu ? cu[s + 1] - cu[s] : single_len;
    int v = (len + bt - 1) / bt;
    nt[s] = v < max_nt ? v : max_nt;  // max_seqlen is a caller-guaranteed bound
  }
  for (int j = t; j < max_nt; j += kPlanThreads) cnt[j] = 0;
  __syncthreads();

  // 2. rank by (tile count desc, index asc); the rank is a permutation
  for (int s = t; s < n; s += kPlanThreads) {
    const int mine = nt[s];
    int rank = 0;
    for (int o = 0; o < n; ++o) {
      const int other = nt[o];
      rank += (other > mine) || (other == mine && o < s);
    }
    order[rank] = s;
  }
  __syncthreads();

  // 3. cnt[j] = number of segments with more than j tiles
  for (int r = t; r < n; r += kPlanThreads) {
    const int hi = nt[order[r]];
    const int lo = (r + 1 < n) ? nt[order[r + 1]] : 0;
    for (int j = lo; j < hi; ++j) cnt[j] = r + 1;
  }
  __syncthreads();

  // 4. start[j] = sum_{j' > j} cnt[j'] (exclusive suffix sum), chunked scan
  const int chunk = (max_nt + kPlanThreads - 1) / kPlanThreads;
  // thread t owns levels counted from the top: idx = t*chunk .. t*chunk+chunk-1,
  // level = max_nt - 1 - idx
  int local = 0;
  for (int c = 0; c < chunk; ++c) {
    const int idx = t * chunk + c;
    if (idx < max_nt) local += cnt[max_nt - 1 - idx];
  }
  part[t] = local;
  __syncthreads();
  if (t == 0) {
    int run = 0;
    for (int i = 0; i < kPlanThreads; ++i) {
      const int v = part[i];
      part[i] = run;
      run += v;
    }
    *total = run;
  }
  __syncthreads();
  int run = part[t];
  for (int c = 0; c < chunk; ++c) {
    const int idx = t * chunk + c;
    if (idx < max_nt) {
      const int j = max_nt - 1 - idx;
      start[j] = run;
      run += cnt[j];
    }
  }
}

}  // namespace pdy
