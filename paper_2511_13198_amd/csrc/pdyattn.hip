// C-ABI of the pdyattn library: argument validation, workspace carving and
// kernel launches.  Declarations and the contract live in include/pdyattn.h.
#include "../../include/pdyattn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <vector>

#include "bwd.hpp"
#include "fwd.hpp"
#include "plan.hpp"

namespace {

thread_local char g_err[512] = "";

pdy_status fail(pdy_status st, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

pdy_status hip_fail(hipError_t e, const char* what) {
  return fail(PDY_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kTile = 128;  // smallest tile of any kernel (bounds the work items)
constexpr int kKvTile = pdy::DkdvCfg<128>::BK;  // keys per dK/dV work item
static_assert(pdy::DkdvCfg<64>::BK == kKvTile, "one key-tile schedule for both head dims");

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

struct Sizes {
  int64_t T, N, maxlen, hq, hkv, d;
  int max_nt;  // tiles of kTile in the longest segment (unused by the launches)
};

int tiles_of(const Sizes& s, int tile) {
  const int64_t n = (s.maxlen + tile - 1) / tile;
  return n < 1 ? 1 : (int)n;
}

// forward and dQ workgroup size: 8 waves (256 query rows, 128-key tiles, one
// workgroup per CU) unless every segment has at most kShortSeg tokens; then
// 4 waves (128 rows, 64-key tiles, two workgroups per CU), whose smaller
// items and diagonal tiles outweigh their extra barriers there (measured
// fwd+bwd: 1K-2K tokens 7-12 % faster, 4K and longer 3-15 % slower)
#ifndef PDY_WAVES_LONG
#define PDY_WAVES_LONG 8
#endif
constexpr int64_t kShortSeg = 2048;
int fwd_waves(const Sizes& s) { return s.maxlen > kShortSeg ? PDY_WAVES_LONG : 4; }

pdy_status check_sizes(int32_t T, int32_t N, int32_t maxlen, int32_t hq, int32_t hkv, int32_t d,
                       Sizes* out) {
  if (T < 0) return fail(PDY_ERR_INVALID_ARG, "total_tokens must be >= 0 (got %d)", T);
  if (N < 1) return fail(PDY_ERR_INVALID_ARG, "num_seqs must be >= 1 (got %d)", N);
  if (maxlen < 0 || maxlen > T)
    return fail(PDY_ERR_INVALID_ARG, "max_seqlen must be in [0, total_tokens] (got %d, T=%d)",
                maxlen, T);
  if (T > 0 && maxlen < 1)
    return fail(PDY_ERR_INVALID_ARG, "max_seqlen must be >= 1 when total_tokens > 0");
  // one segment spans [0, T) by the contract, and a single-segment call
  // builds no tile schedule but sizes its grid from max_seqlen: anything
  // other than T would leave rows unwritten (or visit rows past the end)
  if (N == 1 && maxlen != T)
    return fail(PDY_ERR_INVALID_ARG,
                "with num_seqs = 1 max_seqlen must equal total_tokens (got %d, T=%d)", maxlen, T);
  if (hq < 1 || hkv < 1)
    return fail(PDY_ERR_INVALID_ARG, "head counts must be >= 1 (got Hq=%d, Hkv=%d)", hq, hkv);
  if (hq % hkv != 0)
    return fail(PDY_ERR_INVALID_ARG, "num_heads_q (%d) must be a multiple of num_heads_kv (%d)",
                hq, hkv);
  if (d != 64 && d != 128)
    return fail(PDY_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", d);
  // element offsets are computed in 64 bits; keep T*H*d well inside that and
  // the grid (items x heads) inside 2^31 blocks
  const int64_t items = (int64_t)T / kTile + N;
  if (items * hq >= (int64_t)1 << 31)
    return fail(PDY_ERR_INVALID_ARG, "problem too large for one launch");
  out->T = T;
  out->N = N;
  out->maxlen = maxlen;
  out->hq = hq;
  out->hkv = hkv;
  out->d = d;
  out->max_nt = (int)((maxlen + kTile - 1) / kTile);
  if (out->max_nt < 1) out->max_nt = 1;
  return PDY_OK;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// ---------------------------------------------------------------------------
// Optional per-thread kernel timing: while enabled, every launch is bracketed
// by two events on its own stream; pdy_profile_stop reduces them per kernel.
// ---------------------------------------------------------------------------
enum KernelId { K_PLAN = 0, K_FWD, K_DKDV, K_DQ, K_SPLIT_MERGE, K_SPLIT_SUM, K_COUNT };
const char* const kKernelNames[K_COUNT] = {"plan_kernel",     "fwd_kernel",
                                           "bwd_dkdv_kernel", "bwd_dq_kernel",
                                           "split_merge_kernel", "split_sum_kernel"};
struct ProfRec {
  int kid;
  hipEvent_t a, b;
};
thread_local bool g_prof_on = false;
thread_local std::vector<ProfRec> g_prof_recs;
thread_local std::vector<hipEvent_t> g_prof_pool;

hipError_t prof_event(hipEvent_t* ev) {
  if (!g_prof_pool.empty()) {
    *ev = g_prof_pool.back();
    g_prof_pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(ev);
}

// Launch through `fn` (which enqueues exactly one kernel on `st`), timing it
// when profiling is on.  Returns the launch error, if any.
template <typename F>
hipError_t launch_timed(int kid, hipStream_t st, F fn) {
  if (!g_prof_on) {
    fn();
    return hipGetLastError();
  }
  ProfRec r;
  r.kid = kid;
  hipError_t e = prof_event(&r.a);
  if (e == hipSuccess) e = prof_event(&r.b);
  if (e == hipSuccess) e = hipEventRecord(r.a, st);
  if (e != hipSuccess) return e;
  fn();
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  e = hipEventRecord(r.b, st);
  if (e == hipSuccess) g_prof_recs.push_back(r);
  return e;
}

size_t plan_bytes(const Sizes& s, int tile) {
  return align256(pdy::plan_ints((int)s.N, tiles_of(s, tile)) * 4);
}

size_t dd_bytes(const Sizes& s) { return align256((size_t)s.hq * (size_t)s.T * 4); }

// upper bound on sum_i ceil(len_i / tile) (the number of work items)
int64_t grid_items(const Sizes& s, int tile) {
  const int64_t bound1 = s.T / tile + s.N;
  const int64_t bound2 = s.N * (int64_t)tiles_of(s, tile);
  return bound1 < bound2 ? bound1 : bound2;
}

// Split-K.  A launch whose work items cannot fill the chip (fewer than
// kFillItems workgroups, two per CU) can cut every item's inner loop -- the
// key tiles of a query tile (forward, dQ) or the query steps of a key tile
// (dK/dV) -- into 2 or 4 parts, one workgroup each; the parts' fp32 partial
// results are then combined.  Otherwise the heaviest item alone sets the
// launch's time (a 16K-token sequence over 4 heads has 256 forward items, the
// last of which visits every key).  Splitting shortens the heaviest item by
// (inner - inner/p) tiles but writes and reads back p partial results, so it
// is taken only while that saves time by the estimate below: a tile's time
// from the kernels' measured throughput per CU (≈ 4.5 TFLOP/s forward and
// dK/dV, ≈ 5 dQ), the partial traffic at ≈ 4 TB/s, plus one launch.  The
// decision depends on the sizes alone (balanced_split below also on the
// causal flag), so the workspace queries reproduce it; partial buffers exist
// only for launches this small (parts x items < 2 kFillItems, or at most
// kMaxParts slices of a balanced split of fewer than kCUs workgroups).
constexpr int64_t kFillItems = 512;
constexpr int kMaxSplit = 4;
constexpr double kPartBytesPerUs = 4.0e6;  // partial results written + read back
constexpr double kLaunchUs = 4.0;          // the combining kernel

// inner: tiles of the heaviest item; tile_us: time of one tile; part_bytes:
// bytes of one part's partial results
int split_parts(int64_t items, int64_t inner, double tile_us, double part_bytes) {
  auto saved = [&](int p) {  // estimated time saved by p parts (p = 1: none)
    if (p == 1) return 0.0;
    const int64_t left = (inner + p - 1) / p;
    return (double)(inner - left) * tile_us - (2.0 * p * part_bytes / kPartBytesPerUs + kLaunchUs);
  };
  int p = 1;
  while (p < kMaxSplit && items * p < kFillItems && inner >= 4 * p && saved(2 * p) > saved(p))
    p *= 2;
  return p;
}

int fwd_key_tile(const Sizes& s) {
  const bool w8 = fwd_waves(s) == 8;
  if (s.d == 64) return w8 ? pdy::FwdCfg<64, 8>::BK : pdy::FwdCfg<64, 4>::BK;
  return w8 ? pdy::FwdCfg<128, 8>::BK : pdy::FwdCfg<128, 4>::BK;
}

int dq_key_tile(const Sizes& s) {
  const bool w8 = fwd_waves(s) == 8;
  if (s.d == 64) return w8 ? pdy::DqCfg<64, 8>::BK : pdy::DqCfg<64, 4>::BK;
  return w8 ? pdy::DqCfg<128, 8>::BK : pdy::DqCfg<128, 4>::BK;
}

// microseconds for one CU to process `pairs` (query, key) pairs of one head
// with `flops_per_pair_d` x d FLOPs each at `tflops` per CU
double tile_us(double pairs, const Sizes& s, double flops_per_pair_d, double tflops) {
  return pairs * flops_per_pair_d * (double)s.d / (tflops * 1e6);
}

// A split of `p` parts per item (p = 1: none).
pdy::Split uniform_split(int p) {
  pdy::Split sp{};
  sp.parts = p;
  sp.cap = 0;
  sp.rows = sp.keys = sp.group = 1;
  return sp;
}

constexpr int64_t kCUs = 256;  // compute units of the chip
constexpr int kMaxParts = 16;  // partial slices of a balanced split at most

// Balanced split-K of a causal single-segment launch whose uniform split
// takes p > 1 parts per item.  Under the causal mask the items' units range
// from one to the heaviest item's, so equal part counts leave the heaviest
// item's parts (which set the launch's time) several times the mean part; a
// balanced split gives the heaviest items more parts and light items fewer.
// It is taken only when the uniform split's workgroups fit one round on the
// chip (one per CU): over two rounds the uniform parts, dealt heaviest first,
// already pair a heavy part with a light one on each CU, which balanced parts
// (ordered by item, not by size) do not (8K tokens x 4 heads: 607 against 567
// TFLOP/s).  For a budget of workgroups (over the heads) the smallest cap
// (units per part) that fits it is found by bisection (O(items log units) on
// the host; items < 256 here), with at most kMaxParts slices.  Two budgets
// are tried, the uniform split's workgroup count and one workgroup per CU,
// and the one with the lower estimated time is kept: the heaviest part or the
// mean load per CU, whichever is larger, at unit_us per unit, plus the
// partial results written and read back (slice_bytes for all items of all
// heads) at the rate the uniform split assumes.  `shape` gives kind, nitems,
// total, causal, rows, keys and group.
pdy::Split balanced_split(pdy::Split shape, int p, int64_t heads, double unit_us,
                          double slice_bytes) {
  if ((int64_t)p * shape.nitems * heads > kCUs) return uniform_split(p);
  const int umax = shape.units(0);  // item 0 is the heaviest
  int64_t total_units = 0;
  for (int i = 0; i < shape.nitems; ++i) total_units += shape.units(i);
  const double mean_load = (double)total_units * heads / kCUs;
  auto entries = [&](int cap) {
    int64_t n = 0;
    for (int i = 0; i < shape.nitems; ++i) n += (shape.units(i) + cap - 1) / cap;
    return n * heads;
  };
  auto cap_for = [&](int64_t budget) {
    int lo = std::max(1, (umax + kMaxParts - 1) / kMaxParts), hi = umax;  // umax: one part each
    while (lo < hi) {
      const int mid = (lo + hi) / 2;
      if (entries(mid) <= budget) hi = mid;
      else lo = mid + 1;
    }
    return lo;
  };
  auto est_us = [&](int cap) {
    const double parts_bytes = (double)entries(cap) * slice_bytes / ((double)shape.nitems * heads);
    return std::max((double)cap, mean_load) * unit_us + 2.0 * parts_bytes / kPartBytesPerUs;
  };
  const int64_t b1 = (int64_t)p * shape.nitems * heads;
  int cap = cap_for(b1);
  if (b1 < kCUs) {
    const int cap2 = cap_for(kCUs);
    if (est_us(cap2) < est_us(cap)) cap = cap2;
  }
  shape.cap = cap;
  shape.parts = (umax + cap - 1) / cap;
  return shape.parts > 1 ? shape : uniform_split(1);
}

// workgroups per head of a launch of `items` items (per head) under split sp
int64_t split_entries(const pdy::Split& sp, int64_t items) {
  if (sp.cap == 0) return items * sp.parts;
  int64_t n = 0;
  for (int i = 0; i < sp.nitems; ++i) n += sp.nparts(i);
  return n;
}

// The same split with about half the partial slices (for a fixed-size
// workspace); parts = 1 when nothing is left to split.
pdy::Split halve_split(pdy::Split sp) {
  if (sp.cap == 0) return uniform_split(sp.parts / 2);
  sp.cap *= 2;
  sp.parts = (sp.units(0) + sp.cap - 1) / sp.cap;
  return sp.parts > 1 ? sp : uniform_split(1);
}

// shape of a query-tile launch (forward, dQ) over a single segment
pdy::Split q_shape(const Sizes& s, int causal, int rows, int keys) {
  pdy::Split sp = uniform_split(1);
  sp.kind = 0;
  sp.nitems = tiles_of(s, rows);
  sp.total = (int)s.T;
  sp.causal = causal;
  sp.rows = rows;
  sp.keys = keys;
  return sp;
}

// The split of a launch: none for context-parallel pairs (`chunk`), balanced
// for causal single segments, else uniform.
pdy::Split choose_split(int p, const Sizes& s, int causal, bool chunk, pdy::Split shape,
                        int64_t heads, double unit_us, double slice_bytes) {
  // (a split launch has fewer than 512 items, so a slice holds far fewer than
  // the 2^31 floats the combine kernels index with 32 bits; kept as a guard)
  if (p <= 1 || chunk || slice_bytes / 4 >= 2147483648.0) return uniform_split(1);
  if (s.N == 1 && causal) return balanced_split(shape, p, heads, unit_us, slice_bytes);
  return uniform_split(p);
}

// sq: the query rows' sizes; sk: the keys' (the same for self-attention
// over cu's segments, one chunk each for a context-parallel pair)
pdy::Split fwd_split(const Sizes& sq, const Sizes& sk, int causal, bool chunk) {
  const int rows = 32 * fwd_waves(sq), keys = fwd_key_tile(sq);
  const double unit = tile_us((double)rows * keys, sq, 4.0, 4.5);
  const double slice = (double)sq.T * sq.hq * sq.d * 4;
  const int p = split_parts(grid_items(sq, rows) * sq.hq, tiles_of(sk, keys), unit, slice);
  return choose_split(p, sq, causal, chunk, q_shape(sq, causal, rows, keys), sq.hq, unit, slice);
}

pdy::Split dq_split(const Sizes& sq, const Sizes& sk, int causal, bool chunk) {
  const int rows = 32 * fwd_waves(sq), keys = dq_key_tile(sq);
  const double unit = tile_us((double)rows * keys, sq, 6.0, 5.0);
  const double slice = (double)sq.T * sq.hq * sq.d * 4;
  const int p = split_parts(grid_items(sq, rows) * sq.hq, tiles_of(sk, keys), unit, slice);
  return choose_split(p, sq, causal, chunk, q_shape(sq, causal, rows, keys), sq.hq, unit, slice);
}

// the heaviest key tile visits every 64-row query step of every head of its group
pdy::Split dkdv_split(const Sizes& sq, const Sizes& sk, int causal, bool chunk) {
  const int rows = pdy::DkdvCfg<128>::BQ;
  const int g = (int)(sq.hq / sq.hkv);
  const double unit = tile_us((double)rows * kKvTile, sq, 8.0, 4.5);
  const double slice = 2.0 * sk.T * sk.hkv * sk.d * 4;
  const int p = split_parts(grid_items(sk, kKvTile) * sk.hkv, (int64_t)tiles_of(sq, rows) * g,
                            unit, slice);
  pdy::Split shape = uniform_split(1);
  shape.kind = 1;
  shape.nitems = tiles_of(sk, kKvTile);
  shape.total = (int)sk.T;
  shape.causal = causal;
  shape.rows = rows;
  shape.keys = kKvTile;
  shape.group = g;
  return choose_split(p, sk, causal, chunk || sk.T == 0, shape, sk.hkv, unit, slice);
}

size_t part_o_bytes(const Sizes& s, int p) { return align256((size_t)p * s.T * s.hq * s.d * 4); }
size_t part_lse_bytes(const Sizes& s, int p) { return align256((size_t)p * s.hq * s.T * 4); }
size_t part_kv_bytes(const Sizes& s, int p) { return align256((size_t)p * s.T * s.hkv * s.d * 4); }

// workspace for a split forward's partial O and LSE (none if it is not split)
size_t fwd_split_bytes(const pdy::Split& sp, const Sizes& sq) {
  return sp.parts > 1 ? part_o_bytes(sq, sp.parts) + part_lse_bytes(sq, sp.parts) : 0;
}

// workspace for a split backward's partial dK, dV (key rows) and dQ
size_t bwd_split_bytes(const pdy::Split& kv, const pdy::Split& q, const Sizes& sq,
                       const Sizes& sk) {
  return (kv.parts > 1 ? 2 * part_kv_bytes(sk, kv.parts) : 0) +
         (q.parts > 1 ? part_o_bytes(sq, q.parts) : 0);
}

// workspace of a (non-chunk) backward, causal or not: both tile schedules, D
// and any split-K partials
size_t bwd_workspace_bytes(const Sizes& s) {
  size_t parts = 0;
  for (int causal = 0; causal <= 1; ++causal)
    parts = std::max(parts, bwd_split_bytes(dkdv_split(s, s, causal, false),
                                            dq_split(s, s, causal, false), s, s));
  return plan_bytes(s, kKvTile) + plan_bytes(s, 32 * fwd_waves(s)) + dd_bytes(s) + parts;
}

// A single segment (N = 1: by the contract cu = [0, T], and max_seqlen = T)
// needs no schedule: item i is its level nt - 1 - i, so no plan is built.
bool needs_plan(const Sizes& s) { return s.N > 1; }

// segment-major work order from this many tiles in the longest segment on
constexpr int kSegMajorTiles = 8;

pdy::Plan make_plan(int32_t* ws, const Sizes& s, int tile) {
  const int nt = tiles_of(s, tile);
  pdy::Plan p;
  p.max_nt = nt;
  p.seg_major = nt >= kSegMajorTiles;
  if (!needs_plan(s)) {
    p.order = p.start = p.total = p.cnt = p.before = nullptr;
    return p;
  }
  p.order = ws + s.N;
  p.cnt = ws + 2 * s.N;
  p.start = ws + 2 * s.N + nt;
  p.total = ws + 2 * s.N + 2 * nt;
  p.before = ws + 2 * s.N + 2 * nt + 1;
  return p;
}

template <typename K>
hipError_t set_lds(K kernel, int bytes) {
  return hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                             hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

// One-time per-process kernel attribute setup (LDS above the 64 KiB default).
hipError_t init_kernels() {
  static hipError_t status = [] {
    hipError_t e;
    if ((e = set_lds(pdy::fwd_kernel<64, 4>, pdy::FwdCfg<64, 4>::LDS_BYTES)) != hipSuccess) return e;
    if ((e = set_lds(pdy::fwd_kernel<64, 8>, pdy::FwdCfg<64, 8>::LDS_BYTES)) != hipSuccess) return e;
    if ((e = set_lds(pdy::fwd_kernel<128, 4>, pdy::FwdCfg<128, 4>::LDS_BYTES)) != hipSuccess)
      return e;
    if ((e = set_lds(pdy::fwd_kernel<128, 8>, pdy::FwdCfg<128, 8>::LDS_BYTES)) != hipSuccess)
      return e;
    if ((e = set_lds(pdy::bwd_dkdv_kernel<64>, pdy::DkdvCfg<64>::LDS_BYTES)) != hipSuccess) return e;
    if ((e = set_lds(pdy::bwd_dkdv_kernel<128>, pdy::DkdvCfg<128>::LDS_BYTES)) != hipSuccess)
      return e;
    if ((e = set_lds(pdy::bwd_dq_kernel<64, 4>, pdy::DqCfg<64, 4>::LDS_BYTES)) != hipSuccess)
      return e;
    if ((e = set_lds(pdy::bwd_dq_kernel<64, 8>, pdy::DqCfg<64, 8>::LDS_BYTES)) != hipSuccess)
      return e;
    if ((e = set_lds(pdy::bwd_dq_kernel<128, 4>, pdy::DqCfg<128, 4>::LDS_BYTES)) != hipSuccess)
      return e;
    if ((e = set_lds(pdy::bwd_dq_kernel<128, 8>, pdy::DqCfg<128, 8>::LDS_BYTES)) != hipSuccess)
      return e;
    return hipSuccess;
  }();
  return status;
}

template <int D, int NW>
void launch_fwd(dim3 grid, hipStream_t st, const pdy::FwdArgs& a) {
  using C = pdy::FwdCfg<D, NW>;
  hipLaunchKernelGGL((pdy::fwd_kernel<D, NW>), grid, dim3(C::NT), C::LDS_BYTES, st, a);
}

template <int D, int NW>
void launch_dq(dim3 grid, hipStream_t st, const pdy::BwdArgs& a) {
  using C = pdy::DqCfg<D, NW>;
  hipLaunchKernelGGL((pdy::bwd_dq_kernel<D, NW>), grid, dim3(C::NT), C::LDS_BYTES, st, a);
}

pdy_status check_scale(float scale, int32_t causal) {
  if (causal != 0 && causal != 1) return fail(PDY_ERR_INVALID_ARG, "causal must be 0 or 1");
  if (!std::isfinite(scale) || !(scale > 0.f))
    return fail(PDY_ERR_INVALID_ARG, "scale must be finite and > 0");
  return PDY_OK;
}

pdy_status check_ptr(const void* p, const char* name) {
  if (p == nullptr) return fail(PDY_ERR_INVALID_ARG, "%s is NULL", name);
  if (!aligned16(p)) return fail(PDY_ERR_INVALID_ARG, "%s is not 16-byte aligned", name);
  return PDY_OK;
}

// The schedule of s's segments in tiles of `tile` (cu == nullptr: one segment
// of s.T tokens), written to ws
pdy::PlanJob plan_job(const int32_t* cu, int32_t* ws, const Sizes& s, int tile) {
  return pdy::PlanJob{cu, (int)s.N, tile, tiles_of(s, tile), (int)s.T, ws};
}

// one or two schedules in one launch
pdy_status launch_plans(const pdy::PlanJob& a, const pdy::PlanJob* b, hipStream_t st) {
  pdy::PlanJobs jobs;
  jobs.job[0] = a;
  jobs.job[1] = b ? *b : a;
  const dim3 grid(b ? 2 : 1);
  hipError_t e = launch_timed(K_PLAN, st, [&] {
    hipLaunchKernelGGL(pdy::plan_kernel, grid, dim3(pdy::kPlanThreads), 0, st, jobs);
  });
  if (e != hipSuccess) return hip_fail(e, "plan_kernel launch");
  return PDY_OK;
}

}  // namespace

extern "C" {

const char* pdy_status_string(int32_t status) {
  switch (status) {
    case PDY_OK: return "ok";
    case PDY_ERR_INVALID_ARG: return "invalid argument";
    case PDY_ERR_UNSUPPORTED: return "unsupported configuration";
    case PDY_ERR_WORKSPACE: return "workspace too small";
    case PDY_ERR_HIP: return "HIP runtime error";
    default: return "unknown status";
  }
}

const char* pdy_last_error(void) { return g_err; }

size_t attn_fwd_workspace_size(int32_t T, int32_t N, int32_t maxlen, int32_t hq, int32_t hkv,
                               int32_t d) {
  Sizes s;
  if (check_sizes(T, N, maxlen, hq, hkv, d, &s) != PDY_OK) return 0;
  return plan_bytes(s, 32 * fwd_waves(s)) +
         std::max(fwd_split_bytes(fwd_split(s, s, 0, false), s),
                  fwd_split_bytes(fwd_split(s, s, 1, false), s));
}

size_t attn_bwd_workspace_size(int32_t T, int32_t N, int32_t maxlen, int32_t hq, int32_t hkv,
                               int32_t d) {
  Sizes s;
  if (check_sizes(T, N, maxlen, hq, hkv, d, &s) != PDY_OK) return 0;
  return bwd_workspace_bytes(s);
}

}  // extern "C"

namespace {

// One query chunk against one key/value chunk of the same sequence
// (context-parallel step), or off: rows and keys share cu's segments.
struct Chunk {
  int on = 0;
  int tk = 0;          // key/value rows
  int shift = 0;       // query offset - key offset
  int accumulate = 0;  // backward: add to the gradients instead of writing them
};

pdy_status fwd_impl(const void* q, const void* k, const void* v, const int32_t* cu,
                    const Sizes& s, const Sizes& sk, int32_t causal, float scale, void* o,
                    float* lse,
                    void* workspace, size_t workspace_bytes, void* stream, const Chunk& c,
                    const char* who) {
  pdy_status st;
  const int nw = fwd_waves(s);
  const int tile = 32 * nw;
  // a context-parallel pair does not split: the ring already overlaps its
  // forward calls on two streams, and the backward's partial traffic and
  // extra launches cancel the gain (measured at 131,072 tokens over p = 8)
  const pdy::Split split = fwd_split(s, sk, causal, c.on);
  const int nsplit = split.parts;
  const size_t need = plan_bytes(s, tile) + fwd_split_bytes(split, s);
  if (workspace_bytes < need)
    return fail(PDY_ERR_WORKSPACE, "workspace has %zu bytes, %s needs %zu", workspace_bytes, who,
                need);
  hipError_t e = init_kernels();
  if (e != hipSuccess) return hip_fail(e, "kernel attribute setup");
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  int32_t* ws = reinterpret_cast<int32_t*>(workspace);
  if (needs_plan(s) && (st = launch_plans(plan_job(cu, ws, s, tile), nullptr, hs)) != PDY_OK)
    return st;

  pdy::FwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.cu = cu;
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.plan = make_plan(ws, s, tile);
  a.total_tokens = (int)s.T;
  a.hq = (int)s.hq;
  a.hkv = (int)s.hkv;
  a.causal = causal;
  a.scale_log2 = scale * pdy::kLog2e;
  a.chunked = c.on;
  a.tk = c.tk;
  a.shift = c.shift;
  a.split = split;
  a.part_o = nullptr;
  a.part_lse = nullptr;
  if (nsplit > 1) {
    uint8_t* w = reinterpret_cast<uint8_t*>(workspace) + plan_bytes(s, tile);
    a.part_o = reinterpret_cast<float*>(w);
    a.part_lse = reinterpret_cast<float*>(w + part_o_bytes(s, nsplit));
  }
  const dim3 grid((unsigned)(split_entries(split, grid_items(s, tile)) * s.hq));
  e = launch_timed(K_FWD, hs, [&] {
    if (s.d == 64) {
      if (nw == 8) launch_fwd<64, 8>(grid, hs, a);
      else launch_fwd<64, 4>(grid, hs, a);
    } else {
      if (nw == 8) launch_fwd<128, 8>(grid, hs, a);
      else launch_fwd<128, 4>(grid, hs, a);
    }
  });
  if (e != hipSuccess) return hip_fail(e, "fwd_kernel launch");
  if (nsplit > 1) {
    const size_t threads = (size_t)s.T * s.hq * (s.d / 8);
    const dim3 blocks((unsigned)((threads + 255) / 256));
    e = launch_timed(K_SPLIT_MERGE, hs, [&] {
      uint16_t* out = static_cast<uint16_t*>(o);
      if (s.d == 64)
        hipLaunchKernelGGL(pdy::split_merge_kernel<64>, blocks, dim3(256), 0, hs, a.part_o,
                           a.part_lse, split, out, lse, (int)s.T, (int)s.hq);
      else
        hipLaunchKernelGGL(pdy::split_merge_kernel<128>, blocks, dim3(256), 0, hs, a.part_o,
                           a.part_lse, split, out, lse, (int)s.T, (int)s.hq);
    });
    if (e != hipSuccess) return hip_fail(e, "split_merge_kernel launch");
  }
  return PDY_OK;
}

// sk: sizes of the key side (the query side for self-attention)
size_t bwd_need(const Sizes& s, const Sizes& sk) {
  return plan_bytes(sk, kKvTile) + plan_bytes(s, 32 * fwd_waves(s)) + dd_bytes(s);
}

pdy_status bwd_impl(const void* q, const void* k, const void* v, const void* o, const float* lse,
                    const void* dout, const int32_t* cu, const Sizes& s, const Sizes& sk,
                    int32_t causal, float scale, float* dq, float* dk, float* dv,
                    void* workspace, size_t workspace_bytes, void* stream, const Chunk& c,
                    const char* who, bool fit_splits = false) {
  pdy_status st;
  const int nwq = fwd_waves(s);
  const int qtile = 32 * nwq;
  // (no split-K for a context-parallel pair, as in the forward)
  pdy::Split split_kv = dkdv_split(s, sk, causal, c.on);
  pdy::Split split_q = dq_split(s, sk, causal, c.on);
  // fit_splits: a fixed-size workspace takes fewer split-K parts (the larger
  // partial buffer halved first) when the chosen ones do not fit
  while (fit_splits && bwd_need(s, sk) + bwd_split_bytes(split_kv, split_q, s, sk) >
                           workspace_bytes &&
         (split_kv.parts > 1 || split_q.parts > 1)) {
    const size_t bk = split_kv.parts > 1 ? 2 * part_kv_bytes(sk, split_kv.parts) : 0;
    const size_t bq = split_q.parts > 1 ? part_o_bytes(s, split_q.parts) : 0;
    if (bq >= bk) split_q = halve_split(split_q);
    else split_kv = halve_split(split_kv);
  }
  const int nsplit_kv = split_kv.parts, nsplit_q = split_q.parts;
  const size_t need = bwd_need(s, sk) + bwd_split_bytes(split_kv, split_q, s, sk);
  if (workspace_bytes < need)
    return fail(PDY_ERR_WORKSPACE, "workspace has %zu bytes, %s needs %zu", workspace_bytes, who,
                need);
  hipError_t e = init_kernels();
  if (e != hipSuccess) return hip_fail(e, "kernel attribute setup");
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  int32_t* ws = reinterpret_cast<int32_t*>(workspace);
  int32_t* ws_q = reinterpret_cast<int32_t*>(reinterpret_cast<uint8_t*>(workspace) +
                                              plan_bytes(sk, kKvTile));
  float* dd = reinterpret_cast<float*>(reinterpret_cast<uint8_t*>(workspace) +
                                       plan_bytes(sk, kKvTile) + plan_bytes(s, qtile));

  {
    // the query-tile schedule, and the key-tile one unless there are no keys
    // (the key side has the same segments as the query side, or is a chunk)
    const pdy::PlanJob q_job = plan_job(cu, ws_q, s, qtile);
    const pdy::PlanJob kv_job = plan_job(cu, ws, sk, kKvTile);
    if (needs_plan(s) &&
        (st = launch_plans(q_job, sk.T > 0 ? &kv_job : nullptr, hs)) != PDY_OK)
      return st;
  }
  pdy::BwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = static_cast<const uint16_t*>(o);
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse = lse;
  a.dd = dd;
  a.cu = cu;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.plan = make_plan(ws, sk, kKvTile);
  a.plan_q = make_plan(ws_q, s, qtile);
  a.total_tokens = (int)s.T;
  a.hq = (int)s.hq;
  a.hkv = (int)s.hkv;
  a.causal = causal;
  a.scale = scale;
  a.scale_log2 = scale * pdy::kLog2e;
  a.chunked = c.on;
  a.tk = c.tk;
  a.shift = c.shift;
  a.accumulate = c.accumulate;
  a.split_kv = split_kv;
  a.split_q = split_q;
  a.part_dk = a.part_dv = a.part_dq = nullptr;
  {
    uint8_t* w = reinterpret_cast<uint8_t*>(workspace) + bwd_need(s, sk);
    if (nsplit_kv > 1) {
      a.part_dk = reinterpret_cast<float*>(w);
      a.part_dv = reinterpret_cast<float*>(w + part_kv_bytes(sk, nsplit_kv));
      w += 2 * part_kv_bytes(sk, nsplit_kv);
    }
    if (nsplit_q > 1) a.part_dq = reinterpret_cast<float*>(w);
  }
  // dQ first: it also writes D = rowsum(dO * O), which dK/dV reads
  const dim3 gq((unsigned)(split_entries(split_q, grid_items(s, qtile)) * s.hq));
  e = launch_timed(K_DQ, hs, [&] {
    if (s.d == 64) {
      if (nwq == 8) launch_dq<64, 8>(gq, hs, a);
      else launch_dq<64, 4>(gq, hs, a);
    } else {
      if (nwq == 8) launch_dq<128, 8>(gq, hs, a);
      else launch_dq<128, 4>(gq, hs, a);
    }
  });
  if (e != hipSuccess) return hip_fail(e, "bwd_dq_kernel launch");
  if (sk.T > 0) {
    const dim3 gkv((unsigned)(split_entries(split_kv, grid_items(sk, kKvTile)) * s.hkv));
    e = launch_timed(K_DKDV, hs, [&] {
      if (s.d == 64)
        hipLaunchKernelGGL(pdy::bwd_dkdv_kernel<64>, gkv, dim3(pdy::DkdvCfg<64>::NT),
                           pdy::DkdvCfg<64>::LDS_BYTES, hs, a);
      else
        hipLaunchKernelGGL(pdy::bwd_dkdv_kernel<128>, gkv, dim3(pdy::DkdvCfg<128>::NT),
                           pdy::DkdvCfg<128>::LDS_BYTES, hs, a);
    });
    if (e != hipSuccess) return hip_fail(e, "bwd_dkdv_kernel launch");
  }
  // the parts' partial gradients (dQ, dK, dV), summed in one launch
  pdy::SumJobs jobs{};
  jobs.njobs = 0;
  jobs.accumulate = c.accumulate;
  int64_t sum_blocks = 0;
  auto add_job = [&](const float* parts, float* dst, size_t n, int row_elems,
                     const pdy::Split& sp) {
    const int blocks = (int)((n / 4 + 255) / 256);
    jobs.blocks[jobs.njobs] = blocks;
    jobs.job[jobs.njobs++] = pdy::SumJob{parts, dst, (uint32_t)n, row_elems, sp};
    sum_blocks += blocks;
  };
  if (nsplit_q > 1) add_job(a.part_dq, dq, (size_t)s.T * s.hq * s.d, (int)(s.hq * s.d), split_q);
  if (sk.T > 0 && nsplit_kv > 1) {
    const size_t n = (size_t)sk.T * s.hkv * s.d;
    add_job(a.part_dk, dk, n, (int)(s.hkv * s.d), split_kv);
    add_job(a.part_dv, dv, n, (int)(s.hkv * s.d), split_kv);
  }
  if (jobs.njobs > 0) {
    const dim3 blocks((unsigned)sum_blocks);
    e = launch_timed(K_SPLIT_SUM, hs, [&] {
      hipLaunchKernelGGL(pdy::split_sum_kernel, blocks, dim3(256), 0, hs, jobs);
    });
    if (e != hipSuccess) return hip_fail(e, "split_sum_kernel launch");
  }
  return PDY_OK;
}

// Argument checks of attn_bwd and attn_bwd_noalloc (everything but the
// workspace); s is filled in.  T = 0 passes with PDY_OK before the pointers
// are looked at.
pdy_status bwd_checks(const void* q, const void* k, const void* v, const void* o,
                      const float* lse, const void* dout, const int32_t* cu_seqlens,
                      int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen,
                      int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                      int32_t causal, float scale, float* dq, float* dk, float* dv, Sizes* s) {
  pdy_status st;
  if ((st = check_sizes(total_tokens, num_seqs, max_seqlen, num_heads_q, num_heads_kv, head_dim,
                        s)) != PDY_OK)
    return st;
  if ((st = check_scale(scale, causal)) != PDY_OK) return st;
  if (s->T == 0) return PDY_OK;
  if ((st = check_ptr(q, "q")) || (st = check_ptr(k, "k")) || (st = check_ptr(v, "v")) ||
      (st = check_ptr(o, "o")) || (st = check_ptr(lse, "lse")) ||
      (st = check_ptr(dout, "dout")) || (st = check_ptr(dq, "dq")) ||
      (st = check_ptr(dk, "dk")) || (st = check_ptr(dv, "dv")))
    return st;
  if (cu_seqlens == nullptr) return fail(PDY_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if ((reinterpret_cast<uintptr_t>(cu_seqlens) & 3u) != 0)
    return fail(PDY_ERR_INVALID_ARG, "cu_seqlens is not 4-byte aligned");
  return PDY_OK;
}

// ---------------------------------------------------------------------------
// Static scratch of attn_bwd_noalloc, for callers that cannot allocate.  A
// file-scope device array: every GPU the library runs on holds its own copy
// (kScratchBytes) from the first use until the process ends.  In host code
// `scratch` only names the symbol; its device address on the current device
// comes from hipGetSymbolAddress, looked up once per device and kept.
// Nothing in it has to start at zero: each call writes every scratch entry
// it reads (schedules, D, partial gradients) before reading it.  Calls that
// overlap on one GPU share the array and race.
// ---------------------------------------------------------------------------
constexpr size_t kScratchBytes = (size_t)64 << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch.
pdy_status scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kMaxDevices)
    return fail(PDY_ERR_UNSUPPORTED, "device %d is beyond the %d the scratch table covers", dev,
                kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    if (p == nullptr) return fail(PDY_ERR_HIP, "hipGetSymbolAddress(scratch) returned NULL");
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PDY_OK;
}

// sizes of a chunk: one segment of t tokens
pdy_status chunk_sizes(int32_t tq, int32_t tk, int32_t hq, int32_t hkv, int32_t d, Sizes* sq,
                       Sizes* sk) {
  pdy_status st;
  if (tq < 0 || tk < 0) return fail(PDY_ERR_INVALID_ARG, "chunk lengths must be >= 0");
  if ((st = check_sizes(tq, 1, tq, hq, hkv, d, sq)) != PDY_OK) return st;
  if ((st = check_sizes(tk, 1, tk, hq, hkv, d, sk)) != PDY_OK) return st;
  return PDY_OK;
}

}  // namespace

extern "C" {

pdy_status attn_fwd(const void* q, const void* k, const void* v, const int32_t* cu_seqlens,
                    int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen, int32_t num_heads_q,
                    int32_t num_heads_kv, int32_t head_dim, int32_t causal, float scale, void* o,
                    float* lse, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  Sizes s;
  pdy_status st;
  if ((st = check_sizes(total_tokens, num_seqs, max_seqlen, num_heads_q, num_heads_kv, head_dim,
                        &s)) != PDY_OK)
    return st;
  if ((st = check_scale(scale, causal)) != PDY_OK) return st;
  if (s.T == 0) return PDY_OK;
  if ((st = check_ptr(q, "q")) || (st = check_ptr(k, "k")) || (st = check_ptr(v, "v")) ||
      (st = check_ptr(o, "o")) || (st = check_ptr(lse, "lse")) ||
      (st = check_ptr(workspace, "workspace")))
    return st;
  if (cu_seqlens == nullptr) return fail(PDY_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if ((reinterpret_cast<uintptr_t>(cu_seqlens) & 3u) != 0)
    return fail(PDY_ERR_INVALID_ARG, "cu_seqlens is not 4-byte aligned");
  return fwd_impl(q, k, v, cu_seqlens, s, s, causal, scale, o, lse, workspace, workspace_bytes,
                  stream, Chunk{}, "attn_fwd");
}

size_t attn_fwd_chunk_workspace_size(int32_t tq, int32_t tk, int32_t hq, int32_t hkv, int32_t d) {
  Sizes sq, sk;
  if (chunk_sizes(tq, tk, hq, hkv, d, &sq, &sk) != PDY_OK) return 0;
  return plan_bytes(sq, 32 * fwd_waves(sq));
}

size_t attn_bwd_chunk_workspace_size(int32_t tq, int32_t tk, int32_t hq, int32_t hkv, int32_t d) {
  Sizes sq, sk;
  if (chunk_sizes(tq, tk, hq, hkv, d, &sq, &sk) != PDY_OK) return 0;
  return bwd_need(sq, sk);
}

pdy_status attn_fwd_chunk(const void* q, const void* k, const void* v, int32_t tq, int32_t tk,
                          int32_t q_offset, int32_t k_offset, int32_t num_heads_q,
                          int32_t num_heads_kv, int32_t head_dim, int32_t causal, float scale,
                          void* o, float* lse, void* workspace, size_t workspace_bytes,
                          void* stream) {
  g_err[0] = 0;
  Sizes sq, sk;
  pdy_status st;
  if ((st = chunk_sizes(tq, tk, num_heads_q, num_heads_kv, head_dim, &sq, &sk)) != PDY_OK)
    return st;
  if (q_offset < 0 || k_offset < 0) return fail(PDY_ERR_INVALID_ARG, "offsets must be >= 0");
  if ((st = check_scale(scale, causal)) != PDY_OK) return st;
  if (tq == 0) return PDY_OK;
  if ((st = check_ptr(q, "q")) || (st = check_ptr(o, "o")) || (st = check_ptr(lse, "lse")) ||
      (st = check_ptr(workspace, "workspace")))
    return st;
  if (tk > 0 && ((st = check_ptr(k, "k")) || (st = check_ptr(v, "v")))) return st;
  Chunk c;
  c.on = 1;
  c.tk = tk;
  c.shift = q_offset - k_offset;
  return fwd_impl(q, k, v, nullptr, sq, sk, causal, scale, o, lse, workspace, workspace_bytes, stream,
                  c, "attn_fwd_chunk");
}

pdy_status attn_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
                    const void* dout, const int32_t* cu_seqlens, int32_t num_seqs,
                    int32_t total_tokens, int32_t max_seqlen, int32_t num_heads_q,
                    int32_t num_heads_kv, int32_t head_dim, int32_t causal, float scale, float* dq,
                    float* dk, float* dv, void* workspace, size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  Sizes s;
  pdy_status st;
  if ((st = bwd_checks(q, k, v, o, lse, dout, cu_seqlens, num_seqs, total_tokens, max_seqlen,
                       num_heads_q, num_heads_kv, head_dim, causal, scale, dq, dk, dv, &s)) !=
          PDY_OK ||
      s.T == 0)
    return st;
  if ((st = check_ptr(workspace, "workspace")) != PDY_OK) return st;
  return bwd_impl(q, k, v, o, lse, dout, cu_seqlens, s, s, causal, scale, dq, dk, dv, workspace,
                  workspace_bytes, stream, Chunk{}, "attn_bwd");
}

pdy_status attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o,
                            const float* lse, const void* dout, const int32_t* cu_seqlens,
                            int32_t num_seqs, int32_t total_tokens, int32_t max_seqlen,
                            int32_t num_heads_q, int32_t num_heads_kv, int32_t head_dim,
                            int32_t causal, float scale, float* dq, float* dk, float* dv,
                            void* stream) {
  g_err[0] = 0;
  Sizes s;
  pdy_status st;
  if ((st = bwd_checks(q, k, v, o, lse, dout, cu_seqlens, num_seqs, total_tokens, max_seqlen,
                       num_heads_q, num_heads_kv, head_dim, causal, scale, dq, dk, dv, &s)) !=
          PDY_OK ||
      s.T == 0)
    return st;
  // the scratch attn_bwd takes from its workspace: the tile schedules and D,
  // plus split-K partial gradients where those fit (else fewer parts)
  const size_t need = bwd_need(s, s);
  if (need > kScratchBytes)
    return fail(PDY_ERR_WORKSPACE,
                "attn_bwd_noalloc needs %zu bytes of scratch for these sizes, more than its "
                "static scratch of %zu bytes (call attn_bwd with a workspace instead)",
                need, kScratchBytes);
  void* ws = nullptr;
  if ((st = scratch_ptr(&ws)) != PDY_OK) return st;
  return bwd_impl(q, k, v, o, lse, dout, cu_seqlens, s, s, causal, scale, dq, dk, dv, ws,
                  kScratchBytes, stream, Chunk{}, "attn_bwd_noalloc", /*fit_splits=*/true);
}

pdy_status attn_bwd_chunk(const void* q, const void* k, const void* v, const void* o,
                          const float* lse, const void* dout, int32_t tq, int32_t tk,
                          int32_t q_offset, int32_t k_offset, int32_t num_heads_q,
                          int32_t num_heads_kv, int32_t head_dim, int32_t causal, float scale,
                          float* dq, float* dk, float* dv, int32_t accumulate, void* workspace,
                          size_t workspace_bytes, void* stream) {
  g_err[0] = 0;
  Sizes sq, sk;
  pdy_status st;
  if ((st = chunk_sizes(tq, tk, num_heads_q, num_heads_kv, head_dim, &sq, &sk)) != PDY_OK)
    return st;
  if (q_offset < 0 || k_offset < 0) return fail(PDY_ERR_INVALID_ARG, "offsets must be >= 0");
  if ((st = check_scale(scale, causal)) != PDY_OK) return st;
  if (tq == 0 && tk == 0) return PDY_OK;
  if (tq > 0 && ((st = check_ptr(q, "q")) || (st = check_ptr(o, "o")) ||
                 (st = check_ptr(lse, "lse")) || (st = check_ptr(dout, "dout")) ||
                 (st = check_ptr(dq, "dq"))))
    return st;
  if (tk > 0 && ((st = check_ptr(k, "k")) || (st = check_ptr(v, "v")) ||
                 (st = check_ptr(dk, "dk")) || (st = check_ptr(dv, "dv"))))
    return st;
  if (accumulate != 0 && accumulate != 1)
    return fail(PDY_ERR_INVALID_ARG, "accumulate must be 0 or 1 (got %d)", accumulate);
  if ((st = check_ptr(workspace, "workspace")) != PDY_OK) return st;
  if (tq == 0 && accumulate) return PDY_OK;
  if (tq == 0) {
    // no query rows: the key chunk receives no gradient (a fill kernel, not
    // a memset, so that the call can be captured in a graph)
    hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
    const size_t n = (size_t)tk * num_heads_kv * head_dim;
    const unsigned blocks = (unsigned)((n + 1023) / 1024);
    hipLaunchKernelGGL(pdy::zero_kernel, dim3(blocks), dim3(256), 0, hs, dk, n);
    hipLaunchKernelGGL(pdy::zero_kernel, dim3(blocks), dim3(256), 0, hs, dv, n);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e, "zero_kernel launch");
    return PDY_OK;
  }
  Chunk c;
  c.on = 1;
  c.tk = tk;
  c.shift = q_offset - k_offset;
  c.accumulate = accumulate;
  return bwd_impl(q, k, v, o, lse, dout, nullptr, sq, sk, causal, scale, dq, dk, dv, workspace,
                  workspace_bytes, stream, c, "attn_bwd_chunk");
}

pdy_status attn_merge(const void* o_a, const float* lse_a, const void* o_b, const float* lse_b,
                      int32_t total_tokens, int32_t num_heads_q, int32_t head_dim, void* o,
                      float* lse, void* stream) {
  g_err[0] = 0;
  pdy_status st;
  if (total_tokens < 0) return fail(PDY_ERR_INVALID_ARG, "total_tokens must be >= 0");
  if (num_heads_q < 1) return fail(PDY_ERR_INVALID_ARG, "num_heads_q must be >= 1");
  if (head_dim != 64 && head_dim != 128)
    return fail(PDY_ERR_UNSUPPORTED, "head_dim %d not supported (64 or 128)", head_dim);
  if (total_tokens == 0) return PDY_OK;
  if ((st = check_ptr(o_a, "o_a")) || (st = check_ptr(lse_a, "lse_a")) ||
      (st = check_ptr(o_b, "o_b")) || (st = check_ptr(lse_b, "lse_b")) ||
      (st = check_ptr(o, "o")) || (st = check_ptr(lse, "lse")))
    return st;
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  const size_t threads = (size_t)total_tokens * num_heads_q * (head_dim / 8);
  const unsigned blocks = (unsigned)((threads + 255) / 256);
  const auto* a = static_cast<const uint16_t*>(o_a);
  const auto* b = static_cast<const uint16_t*>(o_b);
  auto* out = static_cast<uint16_t*>(o);
  if (head_dim == 64)
    hipLaunchKernelGGL(pdy::merge_kernel<64>, dim3(blocks), dim3(256), 0, hs, a, lse_a, b, lse_b,
                       out, lse, (int)total_tokens, (int)num_heads_q);
  else
    hipLaunchKernelGGL(pdy::merge_kernel<128>, dim3(blocks), dim3(256), 0, hs, a, lse_a, b, lse_b,
                       out, lse, (int)total_tokens, (int)num_heads_q);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return hip_fail(e, "merge_kernel launch");
  return PDY_OK;
}

pdy_status attn_validate_cu_seqlens(const int32_t* cu_seqlens, int32_t num_seqs,
                                    int32_t total_tokens, int32_t* max_seqlen_out, void* stream) {
  g_err[0] = 0;
  if (cu_seqlens == nullptr) return fail(PDY_ERR_INVALID_ARG, "cu_seqlens is NULL");
  if (num_seqs < 1) return fail(PDY_ERR_INVALID_ARG, "num_seqs must be >= 1");
  std::vector<int32_t> h((size_t)num_seqs + 1);
  hipStream_t hs = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = hipMemcpyAsync(h.data(), cu_seqlens, h.size() * 4, hipMemcpyDeviceToHost, hs);
  if (e == hipSuccess) e = hipStreamSynchronize(hs);
  if (e != hipSuccess) return hip_fail(e, "copying cu_seqlens to the host");
  if (h[0] != 0) return fail(PDY_ERR_INVALID_ARG, "cu_seqlens[0] = %d, expected 0", h[0]);
  int32_t mx = 0;
  for (int32_t i = 0; i < num_seqs; ++i) {
    if (h[i + 1] < h[i])
      return fail(PDY_ERR_INVALID_ARG, "cu_seqlens decreases at %d (%d -> %d)", i, h[i], h[i + 1]);
    if (h[i + 1] - h[i] > mx) mx = h[i + 1] - h[i];
  }
  if (h[num_seqs] != total_tokens)
    return fail(PDY_ERR_INVALID_ARG, "cu_seqlens[%d] = %d, expected total_tokens = %d", num_seqs,
                h[num_seqs], total_tokens);
  if (max_seqlen_out) *max_seqlen_out = mx;
  return PDY_OK;
}

int32_t pdy_kernel_count(void) { return K_COUNT; }

const char* pdy_kernel_name(int32_t k) {
  return (k >= 0 && k < K_COUNT) ? kKernelNames[k] : "";
}

pdy_status pdy_profile_start(void) {
  g_err[0] = 0;
  for (auto& r : g_prof_recs) {
    g_prof_pool.push_back(r.a);
    g_prof_pool.push_back(r.b);
  }
  g_prof_recs.clear();
  g_prof_on = true;
  return PDY_OK;
}

pdy_status pdy_profile_stop(int32_t* launches, double* total_ms, int32_t n) {
  g_err[0] = 0;
  g_prof_on = false;
  if (n < 0 || (n > 0 && (launches == nullptr || total_ms == nullptr)))
    return fail(PDY_ERR_INVALID_ARG, "pdy_profile_stop: bad output arrays");
  for (int32_t k = 0; k < n; ++k) {
    launches[k] = 0;
    total_ms[k] = 0.0;
  }
  pdy_status st = PDY_OK;
  for (auto& r : g_prof_recs) {
    float ms = 0.f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess && st == PDY_OK) st = hip_fail(e, "pdy_profile_stop: reading events");
    if (r.kid < n) {
      launches[r.kid] += 1;
      total_ms[r.kid] += ms;
    }
    g_prof_pool.push_back(r.a);
    g_prof_pool.push_back(r.b);
  }
  g_prof_recs.clear();
  return st;
}

}  // extern "C"
