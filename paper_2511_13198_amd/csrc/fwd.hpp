// Forward of Eq. (2) (section 3): tiled online-softmax attention on the bf16
// matrix cores of gfx950.
//
// One workgroup = one (segment, query head, query tile of 32*NW rows).  With
// NW = 8 two waves share each SIMD, so one wave's softmax (VALU) overlaps the
// other's matrix products.  Each wave owns 32 query rows, with Q held in
// registers as the B operand of
//   S^T = K Q^T            (32 keys x 32 rows per MFMA tile, keys from LDS)
// so that each lane owns one query row (l % 32) and half of the keys of a
// tile; the row max / row sum need one cross-half exchange (permlane32_swap).
// The probabilities are rounded to bf16 and fed back as the B operand of
//   O^T += V^T P^T          (32 head-dim x 32 rows per MFMA tile)
// with V^T read from the row-major LDS tile by transposing reads.  K/V tiles
// (128 keys at d = 128 with 8 waves, else 64) reach LDS by direct copies;
// tile t+1 is in flight while tile t is computed, in softmax steps of 64
// keys.  Tiles entirely above the causal
// diagonal are never visited; only tiles crossing the diagonal or the segment
// end are masked.  When a launch has too few query tiles to fill the chip, a
// workgroup takes one contiguous part of its query tile's key tiles (split-K)
// and writes a partial O and LSE that split_merge_kernel combines.
//
// Softmax statistics are kept in base 2 (log2(e) folded into the scale).  The
// running max used as the exponent offset is only raised when a new tile's max
// exceeds it by more than kRescaleSlack (then the accumulators are rescaled);
// otherwise probabilities up to 2^kRescaleSlack are accumulated as they are.
// The final O = acc / l and LSE = m + log2(l) use the same offset, so the
// result is the same as with exact rescaling at every tile.
#pragma once
#include "common.hpp"

namespace pdy {

constexpr float kRescaleSlack = 8.0f;

#ifndef PDY_FWD_BK
#define PDY_FWD_BK 128
#endif
#ifndef PDY_FWD_STAGES
#define PDY_FWD_STAGES 2
#endif

template <int D, int NW>
struct FwdCfg {
  static constexpr int BQ = 32 * NW;
  // keys per tile (one barrier); 4-wave workgroups keep 64 so that two of
  // them fit a CU's LDS
  static constexpr int BK = (D == 128 && NW == 8) ? PDY_FWD_BK : 64;
  static constexpr int BKS = 64;                            // keys per softmax step
  static constexpr int NT = NW * 64;
  using KL = RowsLayout<D>;  // K is only read as rows
  using VL = DualLayout<D>;  // V is only read transposed
  static constexpr int KTILE = KL::elems(BK);
  static constexpr int VTILE = VL::elems(BK);
  // K/V tiles in flight: the direct copies run STAGES-1 tiles ahead
  static constexpr int STAGES = PDY_FWD_STAGES;
  static constexpr int LDS_BYTES = STAGES * (KTILE + VTILE) * 2;
};

struct FwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* cu;
  uint16_t* o;
  float* lse;
  Plan plan;
  int total_tokens;
  int hq;
  int hkv;
  int causal;
  float scale_log2;  // scale * log2(e)
  // chunk mode (chunked != 0): one query chunk of total_tokens rows over one
  // key/value chunk of tk rows of the same sequence; key j is visible to
  // row i (causal) iff j <= i + shift (shift = query offset - key offset).
  // Otherwise rows and keys share the packed segments of cu.
  int chunked;
  int tk;
  int shift;
  // split-K (split.parts > 1): the key tiles of every query tile are cut into
  // contiguous parts, one workgroup each; part p writes its O (fp32,
  // normalised by its own row sums) to part_o [parts][T][Hq][D] and its LSE
  // to part_lse [parts][Hq][T] instead of o / lse, and split_merge_kernel
  // combines them.  split.parts = 1: o and lse directly.
  Split split;
  float* part_o;
  float* part_lse;
};

// key offset within a 32-key block held in accumulator register r (lane half 0)
__device__ __forceinline__ constexpr int acc_row_off(int r) { return (r >> 2) * 8 + (r & 3); }

// Epilogue of a forward workgroup's wave: normalise its 32 rows and write O
// (bf16) and LSE (natural log), or, for a split-K part, the part's fp32 O and
// LSE.  A row that saw no key (possible for a chunk or a part) gets O = 0 and
// LSE = -inf.  m: the base-2 exponent offset; lsum: this lane's partial row
// sum (the other half of the row's keys is on lane l ^ 32).
template <int D>
__device__ __forceinline__ void fwd_epilogue(const FwdArgs& a, const f32x16 (&oacc)[D / 32],
                                             float m, float lsum, int row, int seg_hi, int h,
                                             int part, int hh) {
  const size_t qstride = (size_t)a.hq * D;
  const float ltot = lsum + partner32(lsum);
  if (row >= seg_hi) return;
  const bool seen = ltot > 0.f;
  const float inv = seen ? 1.f / ltot : 0.f;
  const float lse = seen ? (m + __builtin_log2f(ltot)) * kLn2 : -INFINITY;
  if (a.split.parts > 1) {
    float* op = a.part_o + ((size_t)part * a.total_tokens + row) * qstride + (size_t)h * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 v = {oacc[db][g * 4 + 0] * inv, oacc[db][g * 4 + 1] * inv,
                         oacc[db][g * 4 + 2] * inv, oacc[db][g * 4 + 3] * inv};
        *reinterpret_cast<f32x4*>(op + db * 32 + g * 8 + hh * 4) = v;
      }
    if (hh == 0) a.part_lse[((size_t)part * a.hq + h) * a.total_tokens + row] = lse;
  } else {
    uint16_t* op = a.o + (size_t)row * qstride + (size_t)h * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x2 v01 = {oacc[db][g * 4 + 0] * inv, oacc[db][g * 4 + 1] * inv};
        f32x2 v23 = {oacc[db][g * 4 + 2] * inv, oacc[db][g * 4 + 3] * inv};
        bf16x2 b01 = __builtin_convertvector(v01, bf16x2);
        bf16x2 b23 = __builtin_convertvector(v23, bf16x2);
        u32x2 pk = {__builtin_bit_cast(uint32_t, b01), __builtin_bit_cast(uint32_t, b23)};
        *reinterpret_cast<u32x2*>(op + db * 32 + g * 8 + hh * 4) = pk;
      }
    if (hh == 0) a.lse[(size_t)h * a.total_tokens + row] = lse;
  }
}

template <int D, int NW>
__global__ void __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) fwd_kernel(FwdArgs a) {
  using C = FwdCfg<D, NW>;
  using KL = typename C::KL;
  using VL = typename C::VL;
  constexpr int BQ = C::BQ, BK = C::BK, BKS = C::BKS;
  extern __shared__ __attribute__((aligned(16))) uint16_t smem[];

  // workgroup -> (head, work item, part of its keys), heaviest items first,
  // in the XCD-aware order: the workgroups an XCD runs at a time hold
  // neighbouring query tiles of one head, which stream the same K/V tiles
  // from key 0 and finish close together (4 heads: 1.4 % faster)
  int h, entry, item, part, nparts;
  xcd_order(blockIdx.x, gridDim.x, a.hq, h, entry);
  if (!split_entry(a.split, entry, item, part, nparts)) return;
  int seg, level;
  if (!plan_lookup(a.plan, item, seg, level)) return;
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
  const int row = q0 + w * 32 + (l & 31);  // this lane's query row
  const int wrow0 = q0 + w * 32;
  const int wrow_last = wrow0 + 31;
  // last key this row may see
  const int key_lim = a.causal ? min(row + shift, k_hi - 1) : k_hi - 1;

  const size_t qstride = (size_t)a.hq * D;
  const size_t kvstride = (size_t)a.hkv * D;

  // Q^T as B operand: lane holds Q[row][ks*16 + hh*8 + j]
  bf16x8 qf[D / 16];
  {
    const bool ok = row < seg_hi;
    const uint16_t* qp = a.q + (size_t)row * qstride + (size_t)h * D + hh * 8;
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) qf[ks] = load_bf16x8(qp + ks * 16, ok);
  }

  f32x16 oacc[D / 32];
#pragma unroll
  for (int i = 0; i < D / 32; ++i) oacc[i] = zero16();
  float m = -INFINITY;  // exponent offset (base-2 scaled logits)
  float lsum = 0.f;     // partial row sum over this lane's keys
  f32x16 s[BKS / 32];   // S^T of the keys in flight

  const int kv_end = a.causal ? min(k_hi, q0 + BQ + shift) : k_hi;
  const int ntiles = max(0, (kv_end - k_lo + BK - 1) / BK);
  // this part's key tiles [t_begin, t_end) (possibly none)
  const int t_begin = part * ntiles / nparts;
  const int t_end = (part + 1) * ntiles / nparts;

  auto kbuf = [&](int t) __attribute__((always_inline)) {
    return smem + (t % C::STAGES) * (C::KTILE + C::VTILE);
  };
  auto vbuf = [&](int t) __attribute__((always_inline)) { return kbuf(t) + C::KTILE; };
  const int k_lane = row_lane_base<KL>();
  const int v_lane = tr_lane_base<VL>();
  auto active = [&](int t) __attribute__((always_inline)) {
    return (wrow0 < seg_hi) && (!a.causal || k_lo + t * BK <= wrow_last + shift);
  };

  // S^T for the tile's 32-key blocks; the independent chains interleave
  // S^T for the tile's two 32-key blocks; K fragments are read PIPE k-steps
  // ahead of the products that consume them
  auto compute_s = [&](const uint16_t* ktile, auto&& hook) __attribute__((always_inline)) {
    constexpr int NKS = D / 16, NKB = BKS / 32;
    static_assert(NKB == 2 || NKB == 4, "two or four 32-key blocks per tile");
    constexpr int PIPE = NKB == 2 ? 3 : 1;  // lgkmcnt counts at most 15 reads
    const uint32_t ka = lds_addr(ktile) + k_lane * 2;
    u32x4 kr[PIPE + 1][NKB];
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) s[kb] = zero16();
    auto rd = [&](auto KS) __attribute__((always_inline)) {
      constexpr int ks = decltype(KS)::value, sl = ks % (PIPE + 1);
      static_for<NKB>([&](auto KB) {
        row_issue<KL, decltype(KB)::value * 32, ks * 16>(ka, kr[sl][KB]);
      });
    };
    auto wt = [&](auto KS, auto N) __attribute__((always_inline)) {
      constexpr int sl = decltype(KS)::value % (PIPE + 1);
      if constexpr (NKB == 2) row_wait<decltype(N)::value>(kr[sl][0], kr[sl][1]);
      else row_wait<decltype(N)::value>(kr[sl][0], kr[sl][1], kr[sl][2], kr[sl][3]);
    };
    static_for<PIPE>([&](auto KS) { rd(KS); });
    static_for<NKS>([&](auto KS) {
      constexpr int ks = decltype(KS)::value, slot = ks % (PIPE + 1);
      if constexpr (ks + PIPE < NKS) {
        rd(std::integral_constant<int, ks + PIPE>{});
        wt(KS, std::integral_constant<int, NKB * PIPE>{});
      } else {
        wt(KS, std::integral_constant<int, NKB * (NKS - 1 - ks)>{});
      }
#pragma unroll
      for (int kb = 0; kb < NKB; ++kb) s[kb] = mfma32(as_bf16x8(kr[slot][kb]), qf[ks], s[kb]);
      hook(KS);
    });
  };

  // mask, online softmax, then O^T += V^T P^T
  auto softmax_pv = [&](int k0, const uint16_t* vtile) __attribute__((always_inline)) {
    const bool need_mask = (a.causal && k0 + BKS - 1 > wrow0 + shift) || (k0 + BKS > k_hi);
    if (need_mask) {
#pragma unroll
      for (int kb = 0; kb < BKS / 32; ++kb) {
        const int lim = key_lim - (k0 + kb * 32 + hh * 4);
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (acc_row_off(r) > lim) s[kb][r] = -INFINITY;
      }
    }
    // row max over the lane's 32 logits in four independent chains
    float mx[4] = {-INFINITY, -INFINITY, -INFINITY, -INFINITY};
#pragma unroll
    for (int kb = 0; kb < BKS / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx[r & 3] = fmaxf(mx[r & 3], s[kb][r]);
    float tmax = fmaxf(fmaxf(mx[0], mx[1]), fmaxf(mx[2], mx[3]));
    tmax = fmaxf(tmax, partner32(tmax));
    const float mt = tmax * a.scale_log2;
    const bool grow = mt > m + kRescaleSlack;
    if (__builtin_amdgcn_ballot_w64(grow) != 0) {
      const float alpha = grow ? fast_exp2(m - mt) : 1.f;
      m = grow ? mt : m;
      lsum *= alpha;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
    }
    const float muse = (m == -INFINITY) ? 0.f : m;
    float ps[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kb = 0; kb < BKS / 32; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = fast_exp2(__builtin_fmaf(s[kb][r], a.scale_log2, -muse));
        s[kb][r] = p;
        ps[r & 3] += p;
      }
    lsum += (ps[0] + ps[1]) + (ps[2] + ps[3]);
    // O^T += V^T P^T over the tile's 16-key steps; the transposing reads of
    // step t+1 are in flight while step t multiplies
    constexpr int NDB = D / 32, NT16 = BKS / 16;
    const uint32_t va = lds_addr(vtile) + v_lane * 2;
    TrRegs vr[2][NDB];  // step T uses vr[T & 1]; no copies of in-flight registers
    // priority for the wave while it issues these products, as in the
    // backward's product phases (forward 0.8 % faster; in the S^T products
    // it is 1.6 % slower)
    __builtin_amdgcn_s_setprio(1);
    static_for<NDB>([&](auto DB) { tr_issue<VL, 0, DB * 32>(va, vr[0][DB]); });
    static_for<NT16>([&](auto T) {
      constexpr int cur = T & 1;
      if constexpr (T + 1 < NT16) {
        static_for<NDB>([&](auto DB) { tr_issue<VL, (T + 1) * 16, DB * 32>(va, vr[cur ^ 1][DB]); });
        tr_wait<2 * NDB>(vr[cur]);
      } else {
        tr_wait<0>(vr[cur]);
      }
      const bf16x8 pf = pack8(s[T >> 1], (T & 1) * 8);
#pragma unroll
      for (int db = 0; db < NDB; ++db) oacc[db] = mfma32(vr[cur][db].operand(), pf, oacc[db]);
    });
    __builtin_amdgcn_s_setprio(0);
  };

  const uint16_t* kbase = a.k + (size_t)hk * D;
  const uint16_t* vbase = a.v + (size_t)hk * D;
  // keys past the segment end read as zeros (the copies' range check); they
  // are always masked
  {
    // K/V tiles land in LDS by direct copies, no staging registers
    TileDma<KL, BK, NW> kd;
    TileDma<VL, BK, NW> vd;
    kd.init(kvstride);
    vd.init(kvstride);
    auto issue = [&](int t) __attribute__((always_inline)) {
      const int kt = k_lo + t * BK;
      kd.issue(kbase + (size_t)kt * kvstride, kvstride, k_hi - kt, kbuf(t));
      vd.issue(vbase + (size_t)kt * kvstride, kvstride, k_hi - kt, vbuf(t));
    };
    constexpr int S = C::STAGES;
    constexpr int PK = TileDma<KL, BK, NW>::PER_WAVE, PV = TileDma<VL, BK, NW>::PER_WAVE;
    // copies this wave issues per tile (the fewest over the waves); waiting
    // for "at most (S-2)*kMin outstanding" therefore covers tile it
    constexpr int kMin = TileDma<KL, BK, NW>::INSTS / NW + TileDma<VL, BK, NW>::INSTS / NW;
#pragma unroll
    for (int t = 0; t < S - 1; ++t)
      if (t_begin + t < t_end) issue(t_begin + t);
    for (int it = t_begin; it < t_end; ++it) {
      // tiles it+1 .. it+S-2 may still be in flight
      if (it + S - 2 < t_end) wait_dma_n<(S - 2) * kMin>();
      else wait_dma();
      __syncthreads();
      const int tn = it + S - 1;
      const bool more = tn < t_end;
      if (active(it)) {
        // the copies of tile tn go out one per K-step of S, so that they
        // trickle into the memory pipeline instead of queueing at once;
        // past the last tile they get an empty range (they fetch nothing and
        // fill the free stage with zeros), so that no branch surrounds them
        const int kt = k_lo + tn * BK;
        const int rows_next = more ? k_hi - kt : 0;
        const auto rsk = TileDma<KL, BK, NW>::src(kbase + (size_t)kt * kvstride, kvstride, rows_next);
        const auto rsv = TileDma<VL, BK, NW>::src(vbase + (size_t)kt * kvstride, kvstride, rows_next);
        uint16_t* kl = kbuf(tn);
        uint16_t* vl = vbuf(tn);
        // V's copies first: every wave has the same number of them, while a
        // wave's last K copy may lie past the tile and sits behind a branch,
        // which is then outside the K-steps of S
        auto copy = [&](auto CI) __attribute__((always_inline)) {
          constexpr int c = decltype(CI)::value;
          if constexpr (c < PV) {
            vd.issue_one(c, rsv, vl);
          } else if constexpr (c < PV + PK) {
            kd.issue_one(c - PV, rsk, kl);
          }
        };
        // the tile is taken in softmax steps of BKS keys; the first step
        // issues the copies
        static_for<BK / BKS>([&](auto SUB) {
          constexpr int sub = decltype(SUB)::value;
          const int k0s = k_lo + it * BK + sub * BKS;
          if (sub == 0 || (k0s < kv_end && (!a.causal || k0s <= wrow_last + shift))) {
            compute_s(kbuf(it) + sub * BKS * KL::ROW, [&](auto KS) __attribute__((always_inline)) {
              if constexpr (sub == 0) {
                constexpr int ks = decltype(KS)::value;
                if constexpr (ks < PK + PV - 1) copy(KS);
                // the other copies that every wave has go out with the last
                // K-step
                if constexpr (ks == D / 16 - 1)
                  static_for<PK + PV - 1>([&](auto CI) {
                    if constexpr (decltype(CI)::value >= D / 16) copy(CI);
                  });
              }
            });
            softmax_pv(k0s, vbuf(it) + sub * BKS * VL::ROW);
          }
        });
        // a wave's last K copy (which may lie past the tile: a branch) at
        // the end of the tile
        copy(std::integral_constant<int, PK + PV - 1>{});
      } else if (more) {
        issue(tn);
      }
    }
    // the last tile's empty-range copies land before the workgroup ends
    wait_dma();
  }

  fwd_epilogue<D>(a, oacc, m, lsum, row, seg_hi, h, part, hh);
}

// n floats set to zero, 4 per thread
__global__ void __launch_bounds__(256) zero_kernel(float* __restrict__ p, size_t n) {
  const size_t i = ((size_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
#pragma unroll
  for (int e = 0; e < 4; ++e)
    if (i + e < n) p[i + e] = 0.f;
}

// Combine two partial results of the same query rows (one per key chunk):
//   LSE = log(exp(LSE_a) + exp(LSE_b)),  O = w_a O_a + w_b O_b,
//   w_x = exp(LSE_x - LSE); a part with LSE = -inf has weight 0, and a row
// where both are -inf stays O = 0, LSE = -inf.  One 8-element slice of a
// row and head per thread; the output may alias either input.
template <int D>
__global__ void __launch_bounds__(256) merge_kernel(const uint16_t* oa, const float* la,
                                                    const uint16_t* ob, const float* lb,
                                                    uint16_t* o, float* lse, int total_tokens,
                                                    int hq) {
  constexpr int LANES = D / 8;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t pair = gid / LANES;  // row * hq + head
  const int sub = (int)(gid % LANES);
  if (pair >= (size_t)total_tokens * hq) return;
  const size_t row = pair / hq;
  const int h = (int)(pair % hq);
  const size_t li = (size_t)h * total_tokens + row;
  const float xa = la[li], xb = lb[li];
  const float mx = fmaxf(xa, xb);
  float wa = 0.f, wb = 0.f, l = -INFINITY;
  if (mx != -INFINITY) {
    const float ea = __expf(xa - mx), eb = __expf(xb - mx);
    const float tot = ea + eb;
    wa = ea / tot;
    wb = eb / tot;
    l = mx + __logf(tot);
  }
  const u32x4 va = *reinterpret_cast<const u32x4*>(oa + pair * D + sub * 8);
  const u32x4 vb = *reinterpret_cast<const u32x4*>(ob + pair * D + sub * 8);
  u32x4 out;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f32x2 x = {wa * __uint_as_float(va[i] << 16) + wb * __uint_as_float(vb[i] << 16),
               wa * __uint_as_float(va[i] & 0xffff0000u) + wb * __uint_as_float(vb[i] & 0xffff0000u)};
    out[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
  }
  *reinterpret_cast<u32x4*>(o + pair * D + sub * 8) = out;
  if (sub == 0) lse[li] = l;
}

// Combine the parts of a split-K forward (each over its own key range of
// the same rows; a row has sp.nparts of its query tile), by the same rule as
// merge_kernel:
//   LSE = log sum_p exp(LSE_p),  O = sum_p exp(LSE_p - LSE) O_p,
// parts with LSE = -inf weigh nothing and a row where every part is -inf
// gets O = 0, LSE = -inf.  Parts are fp32, O is rounded to bf16 once.  One
// 8-element slice of a row and head per thread.
template <int D>
__global__ void __launch_bounds__(256) split_merge_kernel(const float* part_o,
                                                          const float* part_lse, Split sp,
                                                          uint16_t* o, float* lse,
                                                          int total_tokens, int hq) {
  constexpr int LANES = D / 8;
  const size_t gid = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
  const size_t pair = gid / LANES;  // row * hq + head
  const int sub = (int)(gid % LANES);
  const size_t rows = (size_t)total_tokens * hq;  // (row, head) pairs per part
  if (pair >= rows) return;
  const size_t row = pair / hq;
  const int h = (int)(pair % hq);
  const size_t li = (size_t)h * total_tokens + row;
  const int nsplit = sp.nparts(sp.item_of((int)row));
  float mx = -INFINITY;
  for (int p = 0; p < nsplit; ++p) mx = fmaxf(mx, part_lse[p * rows + li]);
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  float tot = 0.f;
  if (mx != -INFINITY) {
    for (int p = 0; p < nsplit; ++p) {
      const float w = __expf(part_lse[p * rows + li] - mx);
      tot += w;
      const float* src = part_o + (p * rows + pair) * D + sub * 8;
      const f32x4 x0 = *reinterpret_cast<const f32x4*>(src);
      const f32x4 x1 = *reinterpret_cast<const f32x4*>(src + 4);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        acc[i] += w * x0[i];
        acc[4 + i] += w * x1[i];
      }
    }
  }
  const float inv = tot > 0.f ? 1.f / tot : 0.f;
  u32x4 out;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f32x2 x = {acc[2 * i] * inv, acc[2 * i + 1] * inv};
    out[i] = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
  }
  *reinterpret_cast<u32x4*>(o + pair * D + sub * 8) = out;
  if (sub == 0) lse[li] = tot > 0.f ? mx + __logf(tot) : -INFINITY;
}

}  // namespace pdy
