// Backward of Eq. (2) (section 3), recomputing the probabilities from the
// saved log-sum-exp instead of storing them.  With S = scale * Q K^T,
// P = exp(S - LSE), D_i = <dO_i, O_i>:
//   dV = P^T dO,  dP = dO V^T,  dS = P * (dP - D),  dK = scale * dS^T Q,
//   dQ = scale * dS K.
// Two kernels, in this order:
//   * bwd_dq_kernel     one workgroup per (segment, query head, 32-row-per-wave
//                       tile); mirrors the forward: computes its rows'
//                       D = rowsum(dO * O) (fp32, written to [Hq, T] for the
//                       next kernel), recomputes S^T and dP^T, forms dS^T and
//                       accumulates dQ^T = K^T dS^T.  No atomics.
//   * bwd_dkdv_kernel   one workgroup per (segment, kv head, 256-key tile); a
//                       wave owns 32 keys (K in an LDS tile, V in registers),
//                       keeps their dK^T / dV^T in accumulators, and sweeps
//                       every query head of the group and every 64-row query
//                       step that sees the keys.  Written once, no atomics.
// When a launch cannot fill the chip, a workgroup takes one part of a tile's
// work (split-K) and one split_sum_kernel launch adds the parts' partial
// gradients of both.
// All outputs are deterministic.
#pragma once
#include "common.hpp"
#include "fwd.hpp"  // acc_row_off

namespace pdy {

// One array of split-K partial gradients to sum: dst = (accumulate ? dst :
// 0) + sum_p parts[p * n + i] in part order, where element i belongs to
// query row or key i / row_elems, which has sp.nparts of its item.  A split
// launch has fewer than 512 items of at most 256 rows or keys, so n < 2^31.
struct SumJob {
  const float* parts;  // [sp.parts][n]
  float* dst;          // [n]
  uint32_t n;          // floats (a multiple of 4: a head dimension of 64 or 128 divides it)
  int row_elems;       // floats per query row or key
  Split sp;
};
struct SumJobs {
  SumJob job[3];
  int blocks[3];  // workgroups of each job, one after another in the grid
  int njobs;
  int accumulate;
};

__device__ __forceinline__ void sum_job(const SumJob& b, int block, int accumulate) {
  const uint32_t i = ((uint32_t)block * 256u + threadIdx.x) * 4u;
  if (i >= b.n) return;
  const int nsplit = b.sp.nparts(b.sp.item_of((int)(i / (uint32_t)b.row_elems)));
  f32x4 acc = accumulate ? *reinterpret_cast<const f32x4*>(b.dst + i) : f32x4{0.f, 0.f, 0.f, 0.f};
  for (int p = 0; p < nsplit; ++p)
    acc += *reinterpret_cast<const f32x4*>(b.parts + (size_t)p * b.n + i);
  *reinterpret_cast<f32x4*>(b.dst + i) = acc;
}

// The partial sums of a split-K backward (dQ, and dK and dV) in one launch:
// 4 floats per thread; each workgroup belongs to one job (so the job's
// fields are uniform over it).
__global__ void __launch_bounds__(256) split_sum_kernel(SumJobs jobs) {
  int b = blockIdx.x;
  if (b < jobs.blocks[0]) return sum_job(jobs.job[0], b, jobs.accumulate);
  b -= jobs.blocks[0];
  if (jobs.njobs > 1 && b < jobs.blocks[1]) return sum_job(jobs.job[1], b, jobs.accumulate);
  b -= jobs.blocks[1];
  if (jobs.njobs > 2 && b < jobs.blocks[2]) sum_job(jobs.job[2], b, jobs.accumulate);
}

#ifndef PDY_DQ_BK
#define PDY_DQ_BK 128
#endif
#ifndef PDY_DKDV_PIPE
#define PDY_DKDV_PIPE 2
#endif

struct BwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const uint16_t* dout;
  const float* lse;  // natural log, [Hq, T]
  float* dd;         // D = rowsum(dO * O), [Hq, T]: written by the dQ kernel, read by dK/dV
  const int32_t* cu;
  float* dq;
  float* dk;
  float* dv;
  Plan plan;    // tiles of DkdvCfg::BK keys
  Plan plan_q;  // tiles of DqCfg::BQ query rows
  int total_tokens;
  int hq;
  int hkv;
  int causal;
  float scale;
  float scale_log2;
  // chunk mode (chunked != 0): one query chunk of total_tokens rows against
  // one key/value chunk of tk rows of the same sequence; key j is visible to
  // row i (causal) iff j <= i + shift.  Otherwise rows and keys share the
  // packed segments of cu.
  int chunked;
  int tk;
  int shift;
  int accumulate;  // add to dq/dk/dv instead of overwriting them
  // split-K (split_*.parts > 1): the work of every dK/dV key tile (its query
  // steps) or dQ query tile (its key tiles) is cut into contiguous parts, one
  // workgroup each, and part p writes its scaled partial gradient to
  // part_dk/part_dv [parts][keys][Hkv][D] or part_dq [parts][T][Hq][D]
  // (fp32, never accumulated; keys = tk for a chunk, else T) for
  // split_sum_kernel to add up.
  Split split_kv;
  Split split_q;
  float* part_dk;
  float* part_dv;
  float* part_dq;
};

// dK/dV: one workgroup of 8 waves per (segment, kv head, 256-key tile).  Wave
// w owns keys 32w..32w+31 of the tile alone: its dK^T / dV^T accumulators,
// its V fragments (held in registers as the B operand of dP) and its K rows
// (in an LDS tile, read as the B operand of S).  Every wave sweeps the same
// 64-row query steps, taking each as two 32-row halves, so the Q/dO tile of a
// step is shared by all eight waves and one barrier covers 64 matrix products
// per wave.  Two waves per SIMD let one wave's softmax recomputation overlap
// the other's matrix products.  Under split-K a workgroup takes one
// contiguous part of the tile's query steps and writes partial dK/dV for
// split_sum_kernel.
template <int D>
struct DkdvCfg {
  static constexpr int NW = 8;
  static constexpr int BK = 32 * NW;  // keys per workgroup (32 per wave)
  static constexpr int BQ = 64;       // query rows per step (two halves of 32)
  static constexpr int NT = NW * 64;
  using QL = DualLayout<D>;  // Q and dO: read as rows (S, dP) and transposed (dK, dV)
  using KL = RowsLayout<D>;  // K: read as rows only
  static constexpr int QTILE = QL::elems(BQ);
  static constexpr int KTILE = KL::elems(BK);
  // per stage: Q tile, dO tile, lse2[BQ], D[BQ]
  static constexpr int STAGE = 2 * QTILE * 2 + 2 * BQ * 4;
  static constexpr int LDS_BYTES = 2 * STAGE + KTILE * 2;
  static_assert(LDS_BYTES <= 160 * 1024, "LDS of one CU");
};

template <int D>
__global__ void __launch_bounds__(512) bwd_dkdv_kernel(BwdArgs a) {
  using C = DkdvCfg<D>;
  using QL = typename C::QL;
  using KL = typename C::KL;
  constexpr int BK = C::BK, BQ = C::BQ, NW = C::NW;
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];

  // workgroup -> (kv head, work item, part of its query steps).  A
  // workgroup streams the query rows from its key tile on; the XCD-aware
  // order keeps those of the workgroups running at a time on one XCD within
  // its L2 (with 2 kv heads and plain round-robin, each XCD would stream
  // every fourth key tile's rows: an 8 MB window and 20x the traffic beyond
  // L2)
  int hk, entry, item, part, nparts;
  xcd_order(blockIdx.x, gridDim.x, a.hkv, hk, entry);
  if (!split_entry(a.split_kv, entry, item, part, nparts)) return;
  int seg, level;
  if (!plan_lookup(a.plan, item, seg, level)) return;
  // keys [k_lo, k_hi) (this workgroup: a tile of them), query rows
  // [q_lo, q_hi); causal: key j visible to row i iff j <= i + shift
  const int k_lo = a.chunked ? 0 : a.cu[seg];
  const int k_hi = a.chunked ? a.tk : a.cu[seg + 1];
  const int q_lo = a.chunked ? 0 : k_lo;
  const int q_hi = a.chunked ? a.total_tokens : k_hi;
  const int shift = a.chunked ? a.shift : 0;
  const int nt = (k_hi - k_lo + BK - 1) / BK;
  const int ktile = nt - 1 - level;
  const int k0 = k_lo + ktile * BK;
  const int g = a.hq / a.hkv;

  const int l = __lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int hh = l >> 5;
  const int kw0 = k0 + w * 32;    // first key of this wave
  const int key = kw0 + (l & 31);  // this lane's key
  const size_t qstride = (size_t)a.hq * D;
  const size_t kvstride = (size_t)a.hkv * D;

  f32x16 dka[D / 32], dva[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) {
    dka[i] = zero16();
    dva[i] = zero16();
  }
  // V^T as B operand of dP = dO V^T: lane holds V[key][ks*16 + hh*8 + j]
  // (keys past the segment end are zeros; their gradients are never written)
  bf16x8 vf[D / 16];
  {
    const uint16_t* vp = a.v + (size_t)key * kvstride + (size_t)hk * D + hh * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) vf[ks] = load_bf16x8(vp + ks * 16, key < k_hi);
  }

  uint8_t* const base = reinterpret_cast<uint8_t*>(smem);
  uint16_t* const ktile_s = reinterpret_cast<uint16_t*>(base + 2 * C::STAGE);
  auto qbuf = [&](int b) __attribute__((always_inline)) {
    return reinterpret_cast<uint16_t*>(base + b * C::STAGE);
  };
  auto gbuf = [&](int b) __attribute__((always_inline)) { return qbuf(b) + C::QTILE; };
  auto stats = [&](int b) __attribute__((always_inline)) {
    return reinterpret_cast<float*>(base + b * C::STAGE + 2 * C::QTILE * 2);
  };

  // query rows that can see this key tile
  const int qstart = a.causal ? max(q_lo, k0 - shift) : q_lo;
  const int nqt = max(0, (q_hi - qstart + BQ - 1) / BQ);
  // this part's steps [s_begin, s_begin + nsteps) of the tile's nqt * g
  const int s_begin = part * (nqt * g) / nparts;
  const int nsteps = (part + 1) * (nqt * g) / nparts - s_begin;
  // a step is one BQ-row tile of one query head of the group: the head's
  // tiles from the last row down to the key tile (the causal diagonal comes
  // last), then the next head's; tracked incrementally (no division in the
  // loop).  Top-down, the workgroups an XCD runs at a time, which hold
  // neighbouring key tiles, start on the same rows and stay close, so the
  // rows they stream are shared in L2 (bottom-up they are a few steps apart
  // and drift further with every head: measured 0.8-1.1 % slower)
  struct StepPos {
    int h;   // query head
    int r0;  // first row
  };
  const int r_last = qstart + (nqt - 1) * BQ;
  const StepPos first = nqt > 0 ? StepPos{hk * g + s_begin / nqt, r_last - (s_begin % nqt) * BQ}
                                 : StepPos{hk * g, qstart};
  auto advance = [&](const StepPos& p) __attribute__((always_inline)) {
    return p.r0 > qstart ? StepPos{p.h, p.r0 - BQ} : StepPos{p.h + 1, r_last};
  };

  // threads 0..BQ-1 fetch the LSE of a row, BQ..2BQ-1 its D.  The value is
  // only touched when stored, after the step's products, so the wait for it
  // (which also covers the tile copies issued with it) is not on the
  // critical path.
  float stat = 0.f;
  auto load_stat = [&](const StepPos& p) __attribute__((always_inline)) {
    const int t = threadIdx.x;
    if (t < 2 * BQ) {
      const int r = p.r0 + (t % BQ);
      const bool ok = r < q_hi;
      const size_t idx = (size_t)p.h * a.total_tokens + r;
      stat = ok ? (t < BQ ? a.lse[idx] : a.dd[idx]) : 0.f;
    }
  };
  auto store_stat = [&](int b) __attribute__((always_inline)) {
    const int t = threadIdx.x;
    // a row without any visible key (LSE = -inf) must contribute nothing:
    // +inf makes exp2(s * scale - lse2) vanish for every s
    if (t < 2 * BQ) stats(b)[t] = t < BQ ? (stat == -INFINITY ? INFINITY : stat * kLog2e) : stat;
  };

  const int q_row = row_lane_base<QL>();
  const int q_tr = tr_lane_base<QL>();
  const int k_row = row_lane_base<KL>();

  // Half `hf` (rows 32 hf .. 32 hf + 31) of a step.  Returns false for a wave
  // with nothing to do there; `hook(KS)` runs after the products of K-step KS
  // of S/dP (active waves only)
  auto compute = [&](int step, const StepPos& p, int hf, auto&& hook) __attribute__((always_inline)) {
    const int b = step & 1;
    const uint16_t* qs = qbuf(b);
    const uint16_t* gs = gbuf(b);
    const float* lse_s = stats(b);
    const float* dd_s = lse_s + BQ;
    const int wr0 = p.r0 + hf * 32;  // first row of this half
    const bool active = (kw0 < k_hi) && (wr0 < q_hi) && (!a.causal || wr0 + 31 + shift >= kw0);
    if (!active) return false;
    const bool need_mask = (a.causal && wr0 + shift < kw0 + 31) || (wr0 + 32 > q_hi);
    // S[row][key] = Q K^T and dP[row][key] = dO V^T for the half's 32 rows;
    // the Q, K and dO fragments of a K-step are read PIPE steps ahead
    f32x16 s = zero16(), dp = zero16();
    {
      constexpr int NKS = D / 16, PIPE = PDY_DKDV_PIPE;
      const uint32_t qa = lds_addr(qs) + (q_row + hf * 32 * QL::ROW) * 2;
      const uint32_t ga = lds_addr(gs) + (q_row + hf * 32 * QL::ROW) * 2;
      const uint32_t ka = lds_addr(ktile_s) + (k_row + w * 32 * KL::ROW) * 2;
      u32x4 rq[PIPE + 1], rk[PIPE + 1], rg[PIPE + 1];
      auto rd = [&](auto KS) __attribute__((always_inline)) {
        constexpr int ks = decltype(KS)::value, sl = ks % (PIPE + 1);
        row_issue<QL, 0, ks * 16>(qa, rq[sl]);
        row_issue<KL, 0, ks * 16>(ka, rk[sl]);
        row_issue<QL, 0, ks * 16>(ga, rg[sl]);
      };
      static_for<PIPE>([&](auto KS) { rd(KS); });
      static_for<NKS>([&](auto KS) {
        constexpr int ks = decltype(KS)::value, sl = ks % (PIPE + 1);
        if constexpr (ks + PIPE < NKS) {
          rd(std::integral_constant<int, ks + PIPE>{});
          row_wait<3 * PIPE>(rq[sl], rk[sl], rg[sl]);
        } else {
          row_wait<3 * (NKS - 1 - ks)>(rq[sl], rk[sl], rg[sl]);
        }
        s = mfma32(as_bf16x8(rq[sl]), as_bf16x8(rk[sl]), s);
        dp = mfma32(as_bf16x8(rg[sl]), vf[ks], dp);
        hook(KS);
      });
    }
    if (need_mask) {  // diagonal or segment-end step only
      // causal: key visible to row iff row - (wr0 + hh*4) >= key - shift - (wr0 + hh*4)
      const int rel = a.causal ? key - shift - wr0 - hh * 4 : -32;
      const int rows_left = q_hi - wr0 - hh * 4;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int off = acc_row_off(r);
        if (off < rel || off >= rows_left) s[r] = -INFINITY;
      }
    }
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int rl = hf * 32 + grp * 8 + hh * 4;
      const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse_s + rl);
      const f32x4 d4 = *reinterpret_cast<const f32x4*>(dd_s + rl);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int r = grp * 4 + e;
        const float pv = fast_exp2(__builtin_fmaf(s[r], a.scale_log2, -l4[e]));
        s[r] = pv;
        dp[r] = pv * (dp[r] - d4[e]);  // dS
      }
    }
    // dV^T += dO^T P  and  dK^T += Q^T dS over two 16-row steps; the
    // transposing reads of the next product are in flight during each one
    constexpr int NDB = D / 32;
    const uint32_t ga = lds_addr(gs) + (q_tr + hf * 32 * QL::ROW) * 2;
    const uint32_t qa = lds_addr(qs) + (q_tr + hf * 32 * QL::ROW) * 2;
    TrRegs ra[NDB], rb[NDB];
    // the two waves of a SIMD run the same phases at about the same time;
    // raising the priority of a wave in this product-only phase lets it keep
    // the matrix core fed while the other wave's exponentials fill the
    // vector ALU (measured: dK/dV 2% faster; no gain in the other phase or
    // the other kernels)
    __builtin_amdgcn_s_setprio(1);
    static_for<NDB>([&](auto DB) { tr_issue<QL, 0, DB * 32>(ga, ra[DB]); });
    static_for<NDB>([&](auto DB) { tr_issue<QL, 0, DB * 32>(qa, rb[DB]); });
    const bf16x8 pb0 = pack8(s, 0), sb0 = pack8(dp, 0);
    tr_wait<2 * NDB>(ra);
#pragma unroll
    for (int db = 0; db < NDB; ++db) dva[db] = mfma32(ra[db].operand(), pb0, dva[db]);
    static_for<NDB>([&](auto DB) { tr_issue<QL, 16, DB * 32>(ga, ra[DB]); });
    tr_wait<2 * NDB>(rb);
#pragma unroll
    for (int db = 0; db < NDB; ++db) dka[db] = mfma32(rb[db].operand(), sb0, dka[db]);
    static_for<NDB>([&](auto DB) { tr_issue<QL, 16, DB * 32>(qa, rb[DB]); });
    const bf16x8 pb1 = pack8(s, 8), sb1 = pack8(dp, 8);
    tr_wait<2 * NDB>(ra);
#pragma unroll
    for (int db = 0; db < NDB; ++db) dva[db] = mfma32(ra[db].operand(), pb1, dva[db]);
    tr_wait<0>(rb);
#pragma unroll
    for (int db = 0; db < NDB; ++db) dka[db] = mfma32(rb[db].operand(), sb1, dka[db]);
    __builtin_amdgcn_s_setprio(0);
    return true;
  };

  auto row_ptr = [&](const uint16_t* t, const StepPos& p) __attribute__((always_inline)) {
    return t + (size_t)p.r0 * qstride + (size_t)p.h * D;
  };
  auto rows_valid = [&](const StepPos& p) __attribute__((always_inline)) { return q_hi - p.r0; };

  // The K tile: keys past the segment end read as zeros (the copies' range
  // check); their gradients are never written out.  Query-side rows past the
  // segment end likewise, and are masked.
  {
    {
      TileDma<KL, BK, NW> kd;
      kd.init(kvstride);
      kd.issue(a.k + (size_t)k0 * kvstride + (size_t)hk * D, kvstride, k_hi - k0, ktile_s);
    }
    using QD = TileDma<QL, BQ, NW>;
    constexpr int PQ = QD::PER_WAVE;  // copies of one tile per wave (at most)
    static_assert(2 * PQ <= D / 16, "one copy per K-step of S/dP");
    QD qd;
    qd.init(qstride);
    auto issue = [&](int step, const StepPos& p) __attribute__((always_inline)) {
      qd.issue(row_ptr(a.q, p), qstride, rows_valid(p), qbuf(step & 1));
      qd.issue(row_ptr(a.dout, p), qstride, rows_valid(p), gbuf(step & 1));
    };
    StepPos cur = first;
    if (nsteps > 0) {
      issue(0, cur);
      load_stat(cur);
    }
    for (int step = 0; step < nsteps; ++step) {
      const bool more = step + 1 < nsteps;
      // (past the last step `nxt` is only used for address arithmetic)
      const StepPos nxt = advance(cur);
      // this step's tiles and statistics have landed (they were issued
      // during the previous step); the statistics go to LDS before the barrier
      wait_dma();
      store_stat(step & 1);
      __syncthreads();
      if (more) load_stat(nxt);
      // the next step's copies go out one per K-step of the first half's
      // S/dP, so that they trickle into the memory pipeline instead of
      // stalling every wave at once; past the last step they get an empty
      // range (they fetch nothing and fill the free stage's Q and dO tiles
      // with zeros), so that no branch surrounds them
      const int rvn = more ? rows_valid(nxt) : 0;
      const typename QD::Src rsq = QD::src(row_ptr(a.q, nxt), qstride, rvn);
      const typename QD::Src rsg = QD::src(row_ptr(a.dout, nxt), qstride, rvn);
      const int bn = (step + 1) & 1;
      // every wave has PQ - 1 copies of each tile; a wave's last one may lie
      // past the tile (a branch), so those two go out at the last K-step
      const bool ran = compute(step, cur, 0, [&](auto KS) __attribute__((always_inline)) {
        constexpr int c = decltype(KS)::value;
        if constexpr (c < PQ - 1) {
          qd.issue_one(c, rsq, qbuf(bn));
        } else if constexpr (c < 2 * (PQ - 1)) {
          qd.issue_one(c - (PQ - 1), rsg, gbuf(bn));
        } else if constexpr (c == D / 16 - 1) {
          qd.issue_one(PQ - 1, rsq, qbuf(bn));
          qd.issue_one(PQ - 1, rsg, gbuf(bn));
        }
      });
      if (!ran && more) issue(step + 1, nxt);
      compute(step, cur, 1, [](auto) {});
      cur = nxt;
    }
  }

  // every copy this wave issued has landed before the workgroup ends (a part
  // with no query steps still issued its K copies)
  wait_dma();
  if (key < k_hi) {
    const bool split = a.split_kv.parts > 1;
    const size_t off = (size_t)key * kvstride + (size_t)hk * D;
    const size_t poff = (size_t)part * (a.chunked ? a.tk : a.total_tokens) * kvstride + off;
    float* dkp = split ? a.part_dk + poff : a.dk + off;
    float* dvp = split ? a.part_dv + poff : a.dv + off;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int d0 = db * 32 + grp * 8 + hh * 4;
        f32x4 kv, vv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int r = grp * 4 + e;
          kv[e] = dka[db][r] * a.scale;
          vv[e] = dva[db][r];
        }
        if (a.accumulate && !split) {
          kv += *reinterpret_cast<const f32x4*>(dkp + d0);
          vv += *reinterpret_cast<const f32x4*>(dvp + d0);
        }
        *reinterpret_cast<f32x4*>(dkp + d0) = kv;
        *reinterpret_cast<f32x4*>(dvp + d0) = vv;
      }
  }
}

template <int D, int NW>
struct DqCfg {
  static constexpr int BQ = 32 * NW;
  static constexpr int BK = (NW == 8) ? PDY_DQ_BK : 64;  // keys per tile
  static constexpr int NT = NW * 64;
  using KL = DualLayout<D>;  // K is read as rows (S^T) and transposed (dQ^T)
  using VL = RowsLayout<D>;  // V is read as rows (dP^T)
  static constexpr int KTILE = KL::elems(BK);
  static constexpr int VTILE = VL::elems(BK);
  static constexpr int LDS_BYTES = 2 * (KTILE + VTILE) * 2;
};

template <int D, int NW>
__global__ void __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) bwd_dq_kernel(BwdArgs a) {
  using C = DqCfg<D, NW>;
  using KL = typename C::KL;
  using VL = typename C::VL;
  constexpr int BQ = C::BQ, BK = C::BK;
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];

  // workgroup -> (head, work item, part of its key tiles), in the XCD-aware
  // order, as in the forward
  int h, entry, item, part, nparts;
  xcd_order(blockIdx.x, gridDim.x, a.hq, h, entry);
  if (!split_entry(a.split_q, entry, item, part, nparts)) return;
  int seg, level;
  if (!plan_lookup(a.plan_q, item, seg, level)) return;
  // query rows [seg_lo, seg_hi), keys [k_lo, k_hi); causal: key j visible to
  // row i iff j <= i + shift
  const int seg_lo = a.chunked ? 0 : a.cu[seg];
  const int seg_hi = a.chunked ? a.total_tokens : a.cu[seg + 1];
  const int k_lo = a.chunked ? 0 : seg_lo;
  const int k_hi = a.chunked ? a.tk : seg_hi;
  const int shift = a.chunked ? a.shift : 0;
  const int q0 = seg_lo + level * BQ;
  const int hk = h / (a.hq / a.hkv);

  const int l = __lane_id();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int hh = l >> 5;
  const int row = q0 + w * 32 + (l & 31);
  const int wrow0 = q0 + w * 32;
  const int wrow_last = wrow0 + 31;
  const int key_lim = a.causal ? min(row + shift, k_hi - 1) : k_hi - 1;
  const size_t qstride = (size_t)a.hq * D;
  const size_t kvstride = (size_t)a.hkv * D;

  // Q and dO of the lane's row as B operands; D = <dO, O> of the row from
  // the lane's half of its elements and the partner lane's (l ^ 32)
  bf16x8 qf[D / 16], gf[D / 16];
  float lse2 = 0.f, ddv = 0.f;
  {
    const bool ok = row < seg_hi;
    const size_t roff = (size_t)row * qstride + (size_t)h * D + hh * 8;
    float dsum[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      qf[ks] = load_bf16x8(a.q + roff + ks * 16, ok);
      gf[ks] = load_bf16x8(a.dout + roff + ks * 16, ok);
      const bf16x8 of = load_bf16x8(a.o + roff + ks * 16, ok);
#pragma unroll
      for (int j = 0; j < 8; ++j)
        dsum[j & 3] = __builtin_fmaf((float)of[j], (float)gf[ks][j], dsum[j & 3]);
    }
    ddv = (dsum[0] + dsum[1]) + (dsum[2] + dsum[3]);
    ddv += partner32(ddv);
    if (ok) {
      lse2 = a.lse[(size_t)h * a.total_tokens + row] * kLog2e;
      // a row without any visible key has LSE = -inf and no gradient
      if (lse2 == -INFINITY) lse2 = INFINITY;
      // D of the row for the dK/dV kernel, which runs after this one
      if (hh == 0 && part == 0) a.dd[(size_t)h * a.total_tokens + row] = ddv;
    }
  }
  f32x16 dqa[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) dqa[i] = zero16();

  const int kv_end = a.causal ? min(k_hi, q0 + BQ + shift) : k_hi;
  const int ntiles = max(0, (kv_end - k_lo + BK - 1) / BK);
  // this part's key tiles [t_begin, t_end) (possibly none)
  const int t_begin = part * ntiles / nparts;
  const int t_end = (part + 1) * ntiles / nparts;
  auto kbuf = [&](int t) __attribute__((always_inline)) { return smem + (t & 1) * C::KTILE; };
  auto vbuf = [&](int t) __attribute__((always_inline)) {
    return smem + 2 * C::KTILE + (t & 1) * C::VTILE;
  };
  const int k_row = row_lane_base<KL>();
  const int k_tr = tr_lane_base<KL>();
  const int v_row = row_lane_base<VL>();
  const uint16_t* kbase = a.k + (size_t)hk * D;
  const uint16_t* vbase = a.v + (size_t)hk * D;

  // returns false for a wave with nothing to do on this tile; `hook(N)` runs
  // after the products of the N-th K-step of S^T/dP^T, counted over the
  // tile's 32-key blocks (active waves only)
  auto compute = [&](int it, auto&& hook) __attribute__((always_inline)) {
    const int k0 = k_lo + it * BK;
    const bool active = (wrow0 < seg_hi) && (!a.causal || k0 <= wrow_last + shift);
    if (!active) return false;
    const uint32_t kra = lds_addr(kbuf(it)) + k_row * 2;
    const uint32_t ka = lds_addr(kbuf(it)) + k_tr * 2;
    const uint32_t vra = lds_addr(vbuf(it)) + v_row * 2;
    const bool need_mask = (a.causal && k0 + BK - 1 > wrow0 + shift) || (k0 + BK > k_hi);
    // one 32-key block at a time keeps S^T and dP^T to 32 registers
    static_for<BK / 32>([&](auto KB) {
      constexpr int kb = decltype(KB)::value;
      // S^T and dP^T; the K and V fragments are read PIPE K-steps ahead
      f32x16 s = zero16(), dp = zero16();
      {
        constexpr int NKS = D / 16, PIPE = 2;
        u32x4 rk[PIPE + 1], rv[PIPE + 1];
        auto rd = [&](auto KS) __attribute__((always_inline)) {
          constexpr int ks = decltype(KS)::value, sl = ks % (PIPE + 1);
          row_issue<KL, kb * 32, ks * 16>(kra, rk[sl]);
          row_issue<VL, kb * 32, ks * 16>(vra, rv[sl]);
        };
        static_for<PIPE>([&](auto KS) { rd(KS); });
        static_for<NKS>([&](auto KS) {
          constexpr int ks = decltype(KS)::value, sl = ks % (PIPE + 1);
          if constexpr (ks + PIPE < NKS) {
            rd(std::integral_constant<int, ks + PIPE>{});
            row_wait<2 * PIPE>(rk[sl], rv[sl]);
          } else {
            row_wait<2 * (NKS - 1 - ks)>(rk[sl], rv[sl]);
          }
          s = mfma32(as_bf16x8(rk[sl]), qf[ks], s);
          dp = mfma32(as_bf16x8(rv[sl]), gf[ks], dp);
          hook(std::integral_constant<int, kb * NKS + ks>{});
        });
      }
      if (need_mask) {  // diagonal or segment-end tile only
        const int lim = key_lim - (k0 + kb * 32 + hh * 4);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (acc_row_off(r) > lim) s[r] = -INFINITY;
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float pv = fast_exp2(__builtin_fmaf(s[r], a.scale_log2, -lse2));
        s[r] = pv * (dp[r] - ddv);  // dS^T
      }
      // dQ^T += K^T dS^T for the block's two 16-key steps
      constexpr int NDB = D / 32;
      TrRegs kt0[NDB], kt1[NDB];
      // priority for the wave in this product-only phase, as in the dK/dV
      // kernel (measured: dQ 2.5% faster)
      __builtin_amdgcn_s_setprio(1);
      // all of kt0 is issued before kt1, so "at most 2*NDB outstanding" means
      // kt0 has landed
      const uint32_t kab = ka + kb * 32 * KL::ROW * 2;
      static_for<NDB>([&](auto DB) { tr_issue<KL, 0, DB * 32>(kab, kt0[DB]); });
      static_for<NDB>([&](auto DB) { tr_issue<KL, 16, DB * 32>(kab, kt1[DB]); });
      tr_wait<2 * NDB>(kt0);
      const bf16x8 sb0 = pack8(s, 0);
#pragma unroll
      for (int db = 0; db < NDB; ++db) dqa[db] = mfma32(kt0[db].operand(), sb0, dqa[db]);
      tr_wait<0>(kt1);
      const bf16x8 sb1 = pack8(s, 8);
#pragma unroll
      for (int db = 0; db < NDB; ++db) dqa[db] = mfma32(kt1[db].operand(), sb1, dqa[db]);
      __builtin_amdgcn_s_setprio(0);
    });
    return true;
  };

  // keys past the segment end read as zeros (the copies' range check); they
  // are always masked
  {
    using KD = TileDma<KL, BK, NW>;
    using VD = TileDma<VL, BK, NW>;
    // the next tile's copies go out one every GAP K-steps of S^T/dP^T rather
    // than all at once after the barrier, as in the dK/dV kernel
    constexpr int PK = KD::PER_WAVE, NCOPY = PK + VD::PER_WAVE;
    constexpr int GAP = (BK / 32) * (D / 16) / NCOPY;
    static_assert(GAP >= 1, "one copy per K-step at most");
    KD kd;
    VD vd;
    kd.init(kvstride);
    vd.init(kvstride);
    auto issue = [&](int t) __attribute__((always_inline)) {
      const int kt = k_lo + t * BK;
      kd.issue(kbase + (size_t)kt * kvstride, kvstride, k_hi - kt, kbuf(t));
      vd.issue(vbase + (size_t)kt * kvstride, kvstride, k_hi - kt, vbuf(t));
    };
    // (a chunk can leave a tile without any visible key tile, or with no keys)
    if (t_begin < t_end) issue(t_begin);
    for (int it = t_begin; it < t_end; ++it) {
      const bool more = it + 1 < t_end;
      wait_dma();
      __syncthreads();
      // past the last tile the copies get an empty range (they fetch
      // nothing and fill the free stage with zeros), so that no branch
      // surrounds them; a wave's last V copy may lie past the tile (a
      // branch), so it goes out at the tile's last K-step
      const int kt = k_lo + (it + 1) * BK;
      const int rows_next = more ? k_hi - kt : 0;
      const typename KD::Src rsk = KD::src(kbase + (size_t)kt * kvstride, kvstride, rows_next);
      const typename VD::Src rsv = VD::src(vbase + (size_t)kt * kvstride, kvstride, rows_next);
      const int bn = (it + 1) & 1;
      const bool ran = compute(it, [&](auto N) __attribute__((always_inline)) {
        constexpr int n = decltype(N)::value;
        if constexpr (n % GAP == 0 && n / GAP < PK) {
          kd.issue_one(n / GAP, rsk, kbuf(bn));
        } else if constexpr (n % GAP == 0 && n / GAP < NCOPY - 1) {
          vd.issue_one(n / GAP - PK, rsv, vbuf(bn));
        } else if constexpr (n == (BK / 32) * (D / 16) - 1) {
          vd.issue_one(NCOPY - 1 - PK, rsv, vbuf(bn));
        }
      });
      if (!ran && more) issue(it + 1);
    }
    // the last tile's empty-range copies land before the workgroup ends
    wait_dma();
  }

  if (row < seg_hi) {
    const bool split = a.split_q.parts > 1;
    const size_t off = (size_t)row * qstride + (size_t)h * D;
    float* dqp = split ? a.part_dq + (size_t)part * a.total_tokens * qstride + off : a.dq + off;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int d0 = db * 32 + grp * 8 + hh * 4;
        f32x4 v = {dqa[db][grp * 4] * a.scale, dqa[db][grp * 4 + 1] * a.scale,
                   dqa[db][grp * 4 + 2] * a.scale, dqa[db][grp * 4 + 3] * a.scale};
        if (a.accumulate && !split) v += *reinterpret_cast<const f32x4*>(dqp + d0);
        *reinterpret_cast<f32x4*>(dqp + d0) = v;
      }
  }
}

}  // namespace pdy
