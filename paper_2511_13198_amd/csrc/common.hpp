// Shared device-side building blocks for the gfx950 attention kernels.
//
// Matrix-core conventions (verified lane layouts of the CDNA4 instruction
// v_mfma_f32_32x32x16_bf16, wave64):
//   A (32 x 16): lane l holds A[l % 32][(l / 32) * 8 + j],   j = 0..7
//   B (16 x 32): lane l holds B[(l / 32) * 8 + j][l % 32],   j = 0..7
//   C (32 x 32): lane l holds C[(r / 4) * 8 + (l / 32) * 4 + r % 4][l % 32], r = 0..15
// Every kernel keeps one "owned" index per lane on the C column (l % 32), so
// per-row softmax statistics stay lane-local.  The contraction index of the
// second product in each chain is taken in the permuted order
//   sigma(hh, j) = (j / 4) * 8 + hh * 4 + j % 4      (hh = l / 32)
// which is exactly the order in which a C tile's registers r = 8t..8t+7 list
// their rows; the matching A operand is then fetched from a row-major LDS tile
// with the transposing read ds_read_b64_tr_b16 (see lds_tr_a_operand).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace pdy {

// Fourth word of a raw buffer resource on gfx950 (32-bit data format, no
// swizzle): the value the buffer range check and LDS copies were verified with.
constexpr int kBufferFlags = 0x00020000;

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

// Compile-time loop: f(std::integral_constant<int, I>) for I = 0..N-1.
template <int N, int I = 0, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// LDS byte address of a pointer into shared memory.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)(p);
}

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Value of x held by lane (l ^ 32), via v_permlane32_swap.
__device__ __forceinline__ float partner32(float x) {
  const int l = __lane_id();
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(l < 32 ? r[1] : r[0]);
}

// Pack 8 fp32 values (v[0..7]) into a bf16x8 operand (round to nearest even).
__device__ __forceinline__ bf16x8 pack8(const f32x16& s, int base) {
  bf16x8 out;
#pragma unroll
  for (int j = 0; j < 8; j += 2) {
    f32x2 two = {s[base + j], s[base + j + 1]};
    bf16x2 b = __builtin_convertvector(two, bf16x2);
    out[j] = b[0];
    out[j + 1] = b[1];
  }
  return out;
}

// 16-byte global load of 8 bf16 as an MFMA operand; zero when !valid.
__device__ __forceinline__ bf16x8 load_bf16x8(const uint16_t* p, bool valid) {
  u32x4 raw = {0u, 0u, 0u, 0u};
  if (valid) raw = *reinterpret_cast<const u32x4*>(p);
  return __builtin_bit_cast(bf16x8, raw);
}

// ---------------------------------------------------------------------------
// LDS tile layouts.  A tile holds rows of D bf16 values as 16-byte chunks; all
// offsets below are in bf16 elements.  Two access patterns occur:
//   * row reads (row_issue): a quarter-wave reads the same chunk of 16
//     consecutive rows;
//   * transposing reads (tr_issue): a half-wave reads 4 consecutive rows
//     x 64 consecutive bytes.
// RowsLayout pads rows to D + 8 elements (272 B for D = 128), which makes row
// reads conflict-free.  DualLayout (D = 128) stores row r at 320 r bytes
// shifted by 16 ((r / 4) mod 4) bytes; its bank pattern 4 (r mod 4) +
// (r / 4) mod 4 (in 16-byte units) makes both patterns conflict-free, and in
// both layouts an operand's address is one per-lane base plus an immediate.
// For D = 64 DualLayout falls back to RowsLayout.
// ---------------------------------------------------------------------------
template <int D>
struct RowsLayout {
  static constexpr int ROW = D + 8;                 // elements per stored row
  static constexpr int SLOTS_PER_ROW = ROW * 2 / 16;  // 16-byte slots incl. padding
  __device__ __forceinline__ static int off(int r, int chunk) { return r * ROW + chunk * 8; }
  // offset of a block shift by (r0 rows, c0 elements); r0 % 16 == 0, c0 % 8 == 0
  static constexpr int delta(int r0, int c0) { return r0 * ROW + c0; }
  // transposing read: offset between the two 8-row halves of a 16-row step
  static constexpr int TR_P1 = 8 * ROW;
  static constexpr int elems(int rows) { return rows * ROW; }
  // chunk stored in slot `w` of row r, or -1 for padding
  __device__ __forceinline__ static int chunk_at(int /*r*/, int w) { return w < D / 8 ? w : -1; }
};

template <int D>
struct DualLayout : RowsLayout<D> {};

template <>
struct DualLayout<128> {
  static constexpr int ROW = 160;  // 320-byte pitch
  static constexpr int SLOTS_PER_ROW = 20;
  __device__ __forceinline__ static int off(int r, int chunk) {
    return r * ROW + (((r >> 2) & 3) + chunk) * 8;
  }
  static constexpr int delta(int r0, int c0) { return r0 * ROW + c0; }
  static constexpr int TR_P1 = 8 * ROW + 16;  // +8 rows moves the shift by 2 chunks
  static constexpr int elems(int rows) { return rows * ROW; }
  __device__ __forceinline__ static int chunk_at(int r, int w) {
    const int c = w - ((r >> 2) & 3);
    return (c >= 0 && c < 16) ? c : -1;
  }
};

// Per-lane base (elements) of a row read: row l % 32, chunk l / 32.
template <class L>
__device__ __forceinline__ int row_lane_base() {
  const int l = __lane_id();
  return L::off(l & 31, l >> 5);
}

// Per-lane base (elements) of a transposing read: in each group of 16 lanes,
// lane i addresses row (hh*4 + i/4) and 4 elements starting at column
// (group % 2) * 16 + 4 * (i % 4).
template <class L>
__device__ __forceinline__ int tr_lane_base() {
  const int l = __lane_id();
  const int hh = l >> 5;
  const int g2 = (l >> 4) & 1;
  const int i = l & 15;
  return L::off(hh * 4 + (i >> 2), g2 * 2 + ((i & 3) >> 1)) + (i & 1) * 4;
}

// A operand "X^T" for an LDS tile X[row][col]: lane l gets
//   element j = X[ROW0 + sigma(l/32, j)][COL0 + l % 32],  j = 0..7,
// i.e. 8 rows (in sigma order) of one column, with two ds_read_b64_tr_b16
// (the instruction hands lane i of a 16-lane group element i % 4 of the rows
// addressed by lanes 4e + i/4, e = 0..3), issued with inline assembly so the
// constant part of the address goes into the instruction's offset field.  (The compiler's
// intrinsic for this instruction neither folds offsets nor knows it cannot
// alias in-flight direct-to-LDS copies, and so waits for them.)  The caller
// must wait with tr_wait before using (or copying) the registers.  `lane_addr` = LDS byte
// address of tile + tr_lane_base<L>(); ROW0 % 16 == 0, COL0 % 32 == 0.
struct TrRegs {
  u32x2 lo, hi;
  __device__ __forceinline__ bf16x8 operand() const {
    const bf16x4 blo = __builtin_bit_cast(bf16x4, lo);
    const bf16x4 bhi = __builtin_bit_cast(bf16x4, hi);
    bf16x8 out;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      out[j] = blo[j];
      out[4 + j] = bhi[j];
    }
    return out;
  }
};

template <class L, int ROW0, int COL0>
__device__ __forceinline__ void tr_issue(uint32_t lane_addr, TrRegs& r) {
  constexpr int off0 = L::delta(ROW0, COL0) * 2;
  constexpr int off1 = off0 + L::TR_P1 * 2;
  static_assert(off1 < 65536, "LDS offset out of range");
  // early-clobber outputs: the second read still needs the address register
  // after the first one has been issued (its data arrives asynchronously)
  asm volatile(
      "ds_read_b64_tr_b16 %0, %2 offset:%3\n\t"
      "ds_read_b64_tr_b16 %1, %2 offset:%4"
      : "=&v"(r.lo), "=&v"(r.hi)
      : "v"(lane_addr), "i"(off0), "i"(off1));
}

// Wait until at most N LDS operations of this wave are outstanding; the
// registers passed in are tied to the wait so that no use is scheduled above it.
template <int N>
__device__ __forceinline__ void tr_wait(TrRegs& a, TrRegs& b, TrRegs& c, TrRegs& d) {
  asm volatile("s_waitcnt lgkmcnt(%8)"
               : "+v"(a.lo), "+v"(a.hi), "+v"(b.lo), "+v"(b.hi), "+v"(c.lo), "+v"(c.hi),
                 "+v"(d.lo), "+v"(d.hi)
               : "i"(N));
}
template <int N>
__device__ __forceinline__ void tr_wait(TrRegs& a, TrRegs& b) {
  asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a.lo), "+v"(a.hi), "+v"(b.lo), "+v"(b.hi) : "i"(N));
}
template <int N, int K>
__device__ __forceinline__ void tr_wait(TrRegs (&r)[K]) {
  static_assert(K == 2 || K == 4, "tr_wait handles 2 or 4 operands");
  if constexpr (K == 4) tr_wait<N>(r[0], r[1], r[2], r[3]);
  else tr_wait<N>(r[0], r[1]);
}

// A/B operand whose 8 contraction elements are contiguous in an LDS row:
// element j of lane l comes from row (ROW0 + l % 32), column
// (COL0 + (l/32)*8 + j); ROW0 % 16 == 0, COL0 % 8 == 0.  Issued with inline
// assembly for explicitly pipelined reads; wait with row_wait before use.  `lane_addr` =
// LDS byte address of tile + row_lane_base<L>().
template <class L, int ROW0, int COL0>
__device__ __forceinline__ void row_issue(uint32_t lane_addr, u32x4& r) {
  constexpr int off = L::delta(ROW0, COL0) * 2;
  static_assert(off < 65536, "LDS offset out of range");
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(lane_addr), "i"(off));
}
template <int N>
__device__ __forceinline__ void row_wait(u32x4& a, u32x4& b) {
  asm volatile("s_waitcnt lgkmcnt(%2)" : "+v"(a), "+v"(b) : "i"(N));
}
template <int N>
__device__ __forceinline__ void row_wait(u32x4& a, u32x4& b, u32x4& c) {
  asm volatile("s_waitcnt lgkmcnt(%3)" : "+v"(a), "+v"(b), "+v"(c) : "i"(N));
}
template <int N>
__device__ __forceinline__ void row_wait(u32x4& a, u32x4& b, u32x4& c, u32x4& d) {
  asm volatile("s_waitcnt lgkmcnt(%4)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d) : "i"(N));
}
__device__ __forceinline__ bf16x8 as_bf16x8(const u32x4& r) { return __builtin_bit_cast(bf16x8, r); }

// Direct global -> LDS copy (buffer_load_dwordx4 ... lds: no registers, no LDS
// store instructions) of a [ROWS x D] bf16 tile (D = 64 or 128) into layout
// L.  One instruction moves 64 lanes x 16 B into 1 KB of consecutive LDS (lane l at
// base + 16 l, the base in M0); lane l of instruction k therefore fills 16-byte
// slot 64 k + l of the tile and fetches whichever global chunk the layout
// stores there.  The copies read through a buffer resource over the tile's
// valid rows: the hardware's range check turns rows >= valid_rows into zeros
// (callers mask them), and padding slots get an offset past any range, so
// they fetch nothing.  Per copy this leaves one M0 write and the load, with
// the lane offsets computed once.  Completion is tracked by vmcnt (wait_dma).
template <class L, int ROWS, int NW>
struct TileDma {
  static constexpr int SLOTS = ROWS * L::SLOTS_PER_ROW;
  static constexpr int INSTS = SLOTS / 64;
  static constexpr int PER_WAVE = (INSTS + NW - 1) / NW;
  static_assert(SLOTS % 64 == 0, "tile must fill whole 1 KB copies");
  static constexpr uint32_t kPadOffset = 0x80000000u;  // out of range for every tile
  uint32_t voff[PER_WAVE];  // byte offset of this lane's chunk in each copy
  int wave;                 // this wave's index (wave-uniform)

  __device__ __forceinline__ void init(size_t gstride) {
    const int l = __lane_id();
    wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int slot = (wave + NW * i) * 64 + l;
      const int r = slot / L::SLOTS_PER_ROW;
      const int c = L::chunk_at(r, slot % L::SLOTS_PER_ROW);
      voff[i] = c < 0 ? kPadOffset : (uint32_t)(((size_t)r * gstride + (size_t)c * 8) * 2);
    }
  }
  // Source of one tile: rows [0, min(valid_rows, ROWS)) at gbase.  The
  // values are wave-uniform; passing them through readfirstlane tells the
  // compiler so (it would otherwise wrap each copy in a loop over the
  // distinct values of the lanes).  Built once per tile, used by its copies.
  struct Src {
    uint32_t lo, hi;  // address
    int bytes;        // range of the buffer resource
  };
  __device__ __forceinline__ static Src src(const uint16_t* gbase, size_t gstride, int valid_rows) {
    const int rows = valid_rows < ROWS ? valid_rows : ROWS;
    const uint64_t addr = reinterpret_cast<uint64_t>(gbase);
    return {(uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)addr),
            (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)(addr >> 32)),
            (int)__builtin_amdgcn_readfirstlane((int)((size_t)rows * gstride * 2))};
  }
  __device__ __forceinline__ static void copy(const Src& s, uint32_t voffset, uint16_t* lds) {
    // device pass only: in the host pass the buffer-resource type makes a
    // second kernel's use of the same copy routine fail to instantiate
#if defined(__HIP_DEVICE_COMPILE__)
    const auto rs = __builtin_amdgcn_make_buffer_rsrc(
        reinterpret_cast<void*>(((uint64_t)s.hi << 32) | s.lo), 0, s.bytes, kBufferFlags);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (__attribute__((address_space(3))) void*)lds, 16,
                                             voffset, 0, 0, 0);
#endif
  }
  // Copy i of this wave alone (0 <= i < PER_WAVE, a constant at the call
  // site); a no-op where the wave has no copy i.  Lets a kernel spread its
  // copies over the products of a step instead of queueing them all at once.
  __device__ __forceinline__ void issue_one(int i, const Src& s, uint16_t* lds) const {
    const int k = wave + NW * i;
    // only a wave's last copy can lie past the tile (NW * (PER_WAVE - 1) <
    // INSTS), so the check folds away for the others once i is a constant
    if (INSTS % NW != 0 && i == PER_WAVE - 1 && k >= INSTS) return;  // wave-uniform
    copy(s, voff[i], lds + k * 512);
  }
  // All of this wave's copies of the tile (valid_rows >= 1).
  __device__ __forceinline__ void issue(const uint16_t* gbase, size_t gstride, int valid_rows,
                                        uint16_t* lds) const {
    const Src s = src(gbase, gstride, valid_rows);
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int k = wave + NW * i;
      if (INSTS % NW != 0 && i == PER_WAVE - 1 && k >= INSTS) break;  // wave-uniform
      copy(s, voff[i], lds + k * 512);
    }
  }
};

// Wait until this wave's outstanding direct-to-LDS copies (and any other
// vector-memory loads) have landed.  A workgroup barrier after it publishes
// the tile to every wave.
__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Wait until at most N of this wave's vector-memory loads are outstanding
// (loads complete in issue order, so everything older than the last N is done).
template <int N>
__device__ __forceinline__ void wait_dma_n() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"i"(N) : "memory");
}

// Work schedule built by plan_kernel: items are (segment, level) pairs with
// level j meaning "tile j of the segment" (forward / dQ) or "tile nt-1-j"
// (dK/dV); a higher level is a heavier causal tile.  Two orders of the same
// items:
//   * level-major: by descending level over all segments, so the heaviest
//     tiles of every segment start first;
//   * segment-major: the longest segment's tiles (heaviest first), then the
//     next longest segment's, and so on.  Workgroups that run at the same
//     time then hold neighbouring tiles of one segment, which stream the same
//     rows or keys, so those reads are shared in L2; the heaviest tiles of
//     the longest segments still start first.  Taken when the longest
//     segment has at least 8 tiles (measured on the packed 65,536-token
//     batch of 25 segments, 32 heads: fwd+bwd 682 -> 754 TFLOP/s; packed
//     GQA batches of 9-53 segments +1 to +7 %); with only a few tiles per
//     segment (6,000 segments of at most 300 tokens) level-major keeps the
//     tail shorter (4 % faster there).
// Returns false when `item` is past the end.
struct Plan {
  const int32_t* order;   // segments sorted by tile count, descending [N];
                          // null: a single segment of max_nt tiles (no schedule)
  const int32_t* start;   // first item of each level [max_nt] (level-major)
  const int32_t* total;   // number of items [1]
  const int32_t* cnt;     // segments with more than j tiles [max_nt]
  const int32_t* before;  // first item of the segments with j + 1 tiles [max_nt]
                          // (segment-major)
  int32_t max_nt;
  int32_t seg_major;      // 1: segment-major order
};

// Head and position in that head's work list of workgroup b of a launch of
// n = nheads x (entries per head).  The hardware deals workgroups to the 8
// XCDs round-robin (workgroup b runs on XCD b % 8; each XCD has 32 CUs and
// its own L2), so with head = b % nheads and entry = b / nheads a head is
// spread over 8 / nheads XCDs, each taking every (8 / nheads)-th entry, and
// what the entries running at a time on one XCD stream spreads over a wide
// window.  When nheads divides 8, each of a head's XCDs instead takes 32
// consecutive entries of the head's heaviest-first list at a time (the
// blocks of a head's XCDs run in reverse order every other round, so no XCD
// always gets the lightest block; with 8 heads this is the plain order).
// Measured at 131,072 tokens: dK/dV with 1 kv head -4.7 %, 2 kv heads
// -3.9 %, 4 kv heads -0.3 to -0.8 %; forward and dQ with 4 query heads
// -1.4 % and -0.6 %.  Other head counts keep the plain order.  A bijection
// on [0, n); the last partial round keeps the plain order.
__device__ __forceinline__ void xcd_order(int b, int n, int nheads, int& head, int& entry) {
  constexpr int kXcd = 8, kPer = 32, kRound = kXcd * kPer;
  head = b % nheads;
  entry = b / nheads;
  if (kXcd % nheads != 0 || b >= n / kRound * kRound) return;
  const int g = kXcd / nheads;          // XCDs per head
  const int sub = (b % kXcd) / nheads;  // which of them
  const int s = b / kXcd;               // workgroup index on this XCD
  const int r = s / kPer, q = s % kPer;
  const int blk = (r & 1) ? g - 1 - sub : sub;
  entry = (r * g + blk) * kPer + q;
}

// Split-K of a launch whose work items cannot fill the chip: each item's
// inner loop (its units: the key tiles of a query tile, or the query steps of
// a key tile over the query heads of its group) is cut into contiguous parts,
// one workgroup each, whose partial results a second kernel combines.
//   * uniform (cap == 0): every item in `parts` parts;
//   * balanced (cap > 0, single-segment launches only): item i (the i-th
//     heaviest) in ceil(units(i) / cap) parts, so that light items are not
//     cut into slivers while the heaviest sets the launch's time; `parts` is
//     then the most parts of any item (the number of partial slices).
// A part p of an item with n parts and u units takes units
// [p u / n, (p + 1) u / n).
struct Split {
  int parts;
  int cap;
  int kind;    // 0: items are query tiles of `rows` rows, units key tiles of `keys`
               // 1: items are key tiles of `keys` keys, units steps of `rows` rows
  int nitems;  // items per head (balanced)
  int total;   // tokens of the segment (balanced)
  int causal;
  int rows, keys;
  int group;   // query heads per kv head (kind 1)

  // units of inner work of item i (balanced), i = 0 the heaviest
  __host__ __device__ int units(int i) const {
    if (kind == 0) {
      const int q0 = (nitems - 1 - i) * rows;
      const int kv_end = causal ? (q0 + rows < total ? q0 + rows : total) : total;
      return (kv_end + keys - 1) / keys;
    }
    const int qstart = causal ? i * keys : 0;
    return (total - qstart + rows - 1) / rows * group;
  }
  __host__ __device__ int nparts(int i) const { return cap ? (units(i) + cap - 1) / cap : parts; }
  // item of the query row (kind 0) or key (kind 1) at `pos`
  __host__ __device__ int item_of(int pos) const {
    return kind == 0 ? nitems - 1 - pos / rows : pos / keys;
  }
};

// Item, part and part count of workgroup `entry` (of one head) under split
// sp.  Balanced: the parts of an item are consecutive entries, heavier items
// first; one pass of the wave over the items (a split launch has fewer than
// 512 items) finds the entry's item.  Returns false past the last part.  All
// results are wave-uniform.
__device__ __forceinline__ bool split_entry_scan(const Split& sp, int entry, int& item, int& part,
                                                 int& nparts);
__device__ __forceinline__ bool split_entry(const Split& sp, int entry, int& item, int& part,
                                            int& nparts) {
  bool ok = true;
  if (sp.cap == 0) {
    item = entry / sp.parts;
    part = entry % sp.parts;
    nparts = sp.parts;
  } else {
    ok = split_entry_scan(sp, entry, item, part, nparts);
  }
  // wave-uniform: kept in scalar registers
  item = __builtin_amdgcn_readfirstlane(item);
  part = __builtin_amdgcn_readfirstlane(part);
  nparts = __builtin_amdgcn_readfirstlane(nparts);
  return ok;
}
__device__ __forceinline__ bool split_entry_scan(const Split& sp, int entry, int& item, int& part,
                                                 int& nparts) {
  const int l = __lane_id();
  const int per = (sp.nitems + 63) >> 6;  // items per lane
  int mine = 0;
  for (int k = 0; k < per; ++k) {
    const int i = l * per + k;
    if (i < sp.nitems) mine += sp.nparts(i);
  }
  int incl = mine;  // inclusive prefix sum over the lanes
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int t = __shfl_up(incl, off);
    if (l >= off) incl += t;
  }
  const unsigned long long hit = __ballot(entry >= incl - mine && entry < incl);
  if (hit == 0) return false;
  const int src = __ffsll((long long)hit) - 1;  // the lane whose items hold the entry
  int base = __shfl(incl - mine, src);
  for (int k = 0; k < per; ++k) {
    const int i = src * per + k;
    const int n = sp.nparts(i);
    if (entry < base + n) {
      item = i;
      part = entry - base;
      nparts = n;
      return true;
    }
    base += n;
  }
  return false;
}

__device__ __forceinline__ bool plan_lookup(const Plan& p, int item, int& seg, int& level) {
  if (p.order == nullptr) {  // one segment: item i is its level max_nt - 1 - i
    if (item >= p.max_nt) return false;
    seg = 0;
    level = p.max_nt - 1 - item;
    return true;
  }
  if (item >= *p.total) return false;
  const int32_t* first = p.seg_major ? p.before : p.start;
  // smallest j with first[j] <= item (first is non-increasing in j)
  int lo = 0, hi = p.max_nt - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (first[mid] <= item) hi = mid;
    else lo = mid + 1;
  }
  if (!p.seg_major) {
    level = lo;
    seg = p.order[item - p.start[lo]];
    return true;
  }
  // the segments with v = lo + 1 tiles hold v consecutive items each, from
  // the heaviest tile (level v - 1) down; they are order[cnt[v] ...]
  const int v = lo + 1;
  const int rel = item - first[lo];
  const int g = rel / v;
  level = lo - (rel - g * v);
  seg = p.order[(v < p.max_nt ? p.cnt[v] : 0) + g];
  return true;
}

}  // namespace pdy
