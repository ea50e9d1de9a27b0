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

namespace pdy {

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
// LDS tile layout.  A tile holds rows of D bf16 values as 16-byte chunks.
// For D = 128 a row is exactly 256 bytes (all 64 banks) and chunk c of row r
// is stored at chunk position c ^ swz(r), swz(r) = 4*(r % 4) + (r / 4) % 4.
// That makes both access patterns below conflict-free:
//   * row reads (16 lanes = 16 consecutive rows, one chunk each): swz is a
//     bijection on any 16 consecutive rows aligned to 16;
//   * transposing reads (32 lanes = 4 consecutive rows x 4 consecutive
//     chunks, rows and chunks aligned to 4): the low two bits of the
//     position come from the chunk, the high two from the row.
// For D = 64 rows are padded to 72 elements instead.
// ---------------------------------------------------------------------------
template <int D>
struct LdsTile {
  static constexpr int ROW = (D == 128) ? 128 : D + 8;  // elements per stored row
  __device__ __forceinline__ static int off(int r, int chunk) {
    if constexpr (D == 128) return r * 128 + ((chunk ^ ((r & 3) * 4 + ((r >> 2) & 3))) << 3);
    else return r * ROW + (chunk << 3);
  }
  static constexpr int bytes(int rows) { return rows * ROW * 2; }
};

// A/B operand whose 8 contraction elements are contiguous in an LDS row:
// element j of lane l comes from row (row0 + l % 32), column (col0 + (l/32)*8 + j).
template <int D>
__device__ __forceinline__ bf16x8 lds_row_operand(const uint16_t* tile, int row0, int col0) {
  const int l = __lane_id();
  const uint16_t* p = tile + LdsTile<D>::off(row0 + (l & 31), (col0 >> 3) + (l >> 5));
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const u32x4*>(p));
}

// A operand "X^T" for a row-major LDS tile X[row][col]: lane l gets
//   element j = X[row0 + sigma(l/32, j)][col0 + l % 32],  j = 0..7,
// i.e. 8 rows (in sigma order) of one column.  Two ds_read_b64_tr_b16: in each
// group of 16 lanes, lane i addresses row (base + i/4), 4 columns starting at
// col0 + (group % 2) * 16 + 4 * (i % 4); the instruction hands lane i the
// element (i % 4) of the rows addressed by lanes 4e + i/4, e = 0..3.
// row0 must be a multiple of 16 and col0 a multiple of 32.
template <int D>
__device__ __forceinline__ bf16x8 lds_tr_a_operand(const uint16_t* tile, int row0, int col0) {
  const int l = __lane_id();
  const int hh = l >> 5;
  const int g2 = (l >> 4) & 1;
  const int i = l & 15;
  const int row = row0 + hh * 4 + (i >> 2);
  const int chunk = (col0 >> 3) + g2 * 2 + ((i & 3) >> 1);
  const int sub = (i & 1) * 4;
  const uint16_t* p0 = tile + LdsTile<D>::off(row, chunk) + sub;
  const uint16_t* p1 = tile + LdsTile<D>::off(row + 8, chunk) + sub;
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p0));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p1));
  bf16x4 blo = __builtin_bit_cast(bf16x4, lo);
  bf16x4 bhi = __builtin_bit_cast(bf16x4, hi);
  bf16x8 out;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    out[j] = blo[j];
    out[4 + j] = bhi[j];
  }
  return out;
}

// Cooperative copy of a [rows x D] bf16 tile (rows of global stride
// `gstride` elements) into registers: NT threads, 16 B per thread per step,
// then into an LdsTile<D> layout.
template <int ROWS, int D, int NT>
struct TileLoader {
  static constexpr int CHUNKS_PER_ROW = D / 8;
  static constexpr int TOTAL = ROWS * CHUNKS_PER_ROW;
  static constexpr int STEPS = TOTAL / NT;
  static_assert(TOTAL % NT == 0, "tile must split evenly over the workgroup");
  u32x4 regs[STEPS];

  // Rows >= valid_rows read as zero.
  __device__ __forceinline__ void load(const uint16_t* base, size_t gstride, int valid_rows) {
    const int t = threadIdx.x;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int c = t + s * NT;
      const int row = c / CHUNKS_PER_ROW;
      const int col = (c % CHUNKS_PER_ROW) * 8;
      u32x4 v = {0u, 0u, 0u, 0u};
      if (row < valid_rows) v = *reinterpret_cast<const u32x4*>(base + (size_t)row * gstride + col);
      regs[s] = v;
    }
  }
  // Rows >= valid_rows (valid_rows >= 1) repeat the last valid row instead of
  // reading zeros: no branch per chunk.  Only for tiles whose out-of-range
  // rows the caller masks out (their probabilities are exactly zero).
  __device__ __forceinline__ void load_clamped(const uint16_t* base, size_t gstride,
                                               int valid_rows) {
    const int t = threadIdx.x;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int c = t + s * NT;
      int row = c / CHUNKS_PER_ROW;
      row = row < valid_rows ? row : valid_rows - 1;
      const int col = (c % CHUNKS_PER_ROW) * 8;
      regs[s] = *reinterpret_cast<const u32x4*>(base + (size_t)row * gstride + col);
    }
  }
  __device__ __forceinline__ void store(uint16_t* lds) const {
    const int t = threadIdx.x;
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
      const int c = t + s * NT;
      const int row = c / CHUNKS_PER_ROW;
      const int chunk = c % CHUNKS_PER_ROW;
      *reinterpret_cast<u32x4*>(lds + LdsTile<D>::off(row, chunk)) = regs[s];
    }
  }
};

// Work schedule built by plan_kernel: items are (segment, level) pairs with
// level j meaning "tile j of the segment" (forward / dQ) or "tile nt-1-j"
// (dK/dV); items are ordered by descending level so the heaviest causal tiles
// start first.  Returns false when `item` is past the end.
struct Plan {
  const int32_t* order;  // segments sorted by tile count, descending [N]
  const int32_t* start;  // first item of each level [max_nt]
  const int32_t* total;  // number of items [1]
  int32_t max_nt;
};

__device__ __forceinline__ bool plan_lookup(const Plan& p, int item, int& seg, int& level) {
  if (item >= *p.total) return false;
  // smallest j with start[j] <= item (start is non-increasing in j)
  int lo = 0, hi = p.max_nt - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (p.start[mid] <= item) hi = mid;
    else lo = mid + 1;
  }
  level = lo;
  seg = p.order[item - p.start[lo]];
  return true;
}

}  // namespace pdy
