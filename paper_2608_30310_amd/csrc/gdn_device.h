// Device helpers for the gfx950 GDN kernels: bf16 conversion, hi/lo splitting,
// MFMA wrappers and the k-slot permutation shared by all scan contractions.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace gdn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((__vector_size__(4 * sizeof(float))));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// The command processor hands workgroups to the 8 XCDs round-robin by linear
// index (workgroup b runs on XCD b % 8), and each XCD has its own L2.  The map
// below turns b into a logical index such that every XCD receives one
// contiguous range of logical indices, so workgroups that are logically
// adjacent (and read the same records) share an L2.  It is a bijection on
// [0, total) whatever the hardware order, so correctness never depends on it.
constexpr int kXcds = 8;
__device__ __forceinline__ int xcd_remap(int b, int total) {
  const int x = b % kXcds, i = b / kXcds;
  const int per = total / kXcds, rem = total % kXcds;
  return x < rem ? x * (per + 1) + i : rem * (per + 1) + (x - rem) * per + i;
}

// The same for a grid of clusters of `cs` consecutive logical units (total a
// multiple of cs): each cluster goes whole to one XCD (its units share records
// in that XCD's L2) and consecutive clusters go to consecutive XCDs, so every
// XCD gets an even share of every part of the grid; a varlen batch's long
// sequences are spread over all XCDs instead of landing on one.  Clusters past
// the last full round of kXcds fall back to xcd_remap.  A bijection on
// [0, total).
__device__ __forceinline__ int xcd_cluster_remap(int b, int total, int cs) {
  const int full = total / (kXcds * cs) * (kXcds * cs);
  if (b >= full) return full + xcd_remap(b - full, total - full);
  const int x = b % kXcds, i = b / kXcds;
  return (kXcds * (i / cs) + x) * cs + i % cs;
}

// Barrier for data exchanged through LDS: waits for this wave's LDS accesses
// only (not for its outstanding global loads, DMA or stores, as
// __syncthreads does), and keeps the compiler from moving memory accesses
// across it.
__device__ __forceinline__ void lds_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ---------------------------------------------------------------- bf16
__device__ __forceinline__ uint16_t f2bf(float x) {
  // round to nearest, ties to even (finite values)
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
__device__ __forceinline__ float bf2f(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}

// x = hi + lo with hi = bf16(x), lo = bf16(x - hi): |x - hi - lo| <= 2^-16 |x|.
__device__ __forceinline__ void split_bf16(float x, uint16_t& hi, uint16_t& lo) {
  hi = f2bf(x);
  lo = f2bf(x - bf2f(hi));
}

// A fragment split into bf16 high and low parts.
struct Frag {
  bf16x8 hi;
  bf16x8 lo;
};

// Split of eight values with the hardware bf16 conversion: hi = bf16(x),
// lo = bf16(x - hi).  The conversion's rounding only moves weight between hi
// and lo; the pair still carries x to ~2^-16 relative.  Per pair of values:
// one packed conversion for hi, the two hi values back as fp32 by a shift and
// a mask of the packed word, two subtractions, one packed conversion for lo.
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ Frag split8(const float (&v)[8]) {
  u32x4 hi, lo;
#pragma unroll
  for (int p = 0; p < 4; ++p) {
    const f32x2 x = {v[2 * p], v[2 * p + 1]};
    const uint32_t h = __builtin_bit_cast(uint32_t, __builtin_convertvector(x, bf16x2));
    const f32x2 d = {x[0] - __uint_as_float(h << 16), x[1] - __uint_as_float(h & 0xFFFF0000u)};
    hi[p] = h;
    lo[p] = __builtin_bit_cast(uint32_t, __builtin_convertvector(d, bf16x2));
  }
  Frag f;
  f.hi = __builtin_bit_cast(bf16x8, hi);
  f.lo = __builtin_bit_cast(bf16x8, lo);
  return f;
}

// Transposing LDS read (ds_read_b64_tr_b16): within each group of 16 lanes,
// the lanes' 8-byte rows X[lane][0..3] form a 16 x 4 matrix of 16-bit values
// and lane i receives X[i/4 + 4j][i%4], j = 0..3.
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4* lds_s16x4_ptr_t;
__device__ __forceinline__ u32x2 lds_read_tr16(const void* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4_ptr_t)p);
  return __builtin_bit_cast(u32x2, v);
}

// Reinterpret two 8-byte halves (4 bf16 each) as one operand.
__device__ __forceinline__ bf16x8 join_halves(u32x2 a, u32x2 b) {
  u32x4 u = u32x4{a.x, a.y, b.x, b.y};
  return __builtin_bit_cast(bf16x8, u);
}

// ---------------------------------------------------------------- MFMA
// D(16x16) += A(16x32) B(32x16), bf16 inputs, fp32 accumulate.  Lane l supplies
// A[l%16][8(l/16)+j] and B[8(l/16)+j][l%16] for j = 0..7 and holds
// D[4(l/16)+i][l%16] for i = 0..3.
__device__ __forceinline__ f32x4 mma(bf16x8 a, bf16x8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

// exact bf16 A times split B: two passes.
__device__ __forceinline__ f32x4 mma_x2(bf16x8 a, const Frag& b, f32x4 c) {
  c = mma(a, b.hi, c);
  return mma(a, b.lo, c);
}

// split A times split B: three passes (the lo*lo term, ~2^-16 relative, is dropped).
__device__ __forceinline__ f32x4 mma_x3(const Frag& a, const Frag& b, f32x4 c) {
  c = mma(a.hi, b.hi, c);
  c = mma(a.hi, b.lo, c);
  return mma(a.lo, b.hi, c);
}

// A operand that is exact bf16 (SPLIT = false) or split (SPLIT = true).
template <bool SPLIT>
__device__ __forceinline__ f32x4 mma_a(const Frag& a, const Frag& b, f32x4 c) {
  if constexpr (SPLIT) return mma_x3(a, b, c);
  else return mma_x2(a.hi, b, c);
}

// split A times a B operand that is exact bf16 (SPLIT = false) or split.
template <bool SPLIT>
__device__ __forceinline__ f32x4 mma_b(const Frag& a, const Frag& b, f32x4 c) {
  if constexpr (SPLIT) return mma_x3(a, b, c);
  c = mma(a.hi, b.hi, c);
  return mma(a.lo, b.hi, c);
}

// ---------------------------------------------------------------- K record lane order
// Position of lane l's 16 bytes inside a K-record fragment: within each
// quarter of 16 lanes the positions are rotated by 4 x the quarter, so the
// 16-byte operand reads (16 consecutive lanes of one quarter) still touch 16
// different bank groups, while the transposing reads of K^T (lanes 16 q + 4 g
// + m of four quarters q at once) spread over twice as many bank groups as
// without the rotation.
__device__ __forceinline__ int kslot(int l) { return (l & 48) | ((l + 4 * (l >> 4)) & 15); }
// The lane whose 16 bytes sit at position p (the inverse of kslot).
__device__ __forceinline__ int kslot_inv(int p) { return (p & 48) | ((p + 16 - 4 * (p >> 4)) & 15); }

// ---------------------------------------------------------------- state row order
// The scan holds the state M (d_k x d_v) in MFMA accumulator tiles of 16 rows.
// Lane (g, c) holds rows 4g..4g+3 of tile td, which are state rows
// strow(td, g, 0..3): within each 32-row k step the tiles' rows are
// interleaved so that the 8 rows a lane holds for a k step (tiles 2 kk and
// 2 kk + 1) are the consecutive rows 32 kk + 8 g .. +7.  Then the contraction
// slots of K M0 (and of (Q M0)^T) hit consecutive key (query) columns, and a
// lane's operand is sixteen consecutive bytes of one key row.
__device__ __forceinline__ int strow(int td, int g, int i) { return 32 * (td >> 1) + 8 * g + 4 * (td & 1) + i; }

// ---------------------------------------------------------------- k-slot permutation
// Within a 32-wide k step, MFMA slot 8g + j (g = lane/16, j = 0..7) is mapped to
// contraction index 4g + j for j < 4 and 16 + 4g + (j - 4) for j >= 4.  With this
// order the accumulator that lane (g, c) holds for two consecutive 16-row tiles,
// rows 4g..4g+3 of each, is exactly its B operand for the next contraction over
// those 32 rows, so results chain through registers without a shuffle.
__device__ __forceinline__ int kperm(int g, int j) { return (j < 4) ? 4 * g + j : 16 + 4 * g + (j - 4); }

// B fragment over rows [32kk, 32kk + 32) from two accumulator tiles (rows
// 32kk..32kk+15 and 32kk+16..32kk+31), optionally scaled per element.
__device__ __forceinline__ Frag chain_frag(const f32x4& lo_tile, const f32x4& hi_tile) {
  float v[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    v[j] = lo_tile[j];
    v[4 + j] = hi_tile[j];
  }
  return split8(v);
}

__device__ __forceinline__ f32x4 zero4() {
  f32x4 z = {0.f, 0.f, 0.f, 0.f};
  return z;
}

// ---------------------------------------------------------------- element access
// Raw storage bits of an element (bf16 bits or fp32 bits) and their value.
__device__ __forceinline__ uint32_t load_bits(const float* p, int64_t i) { return __float_as_uint(p[i]); }
__device__ __forceinline__ uint32_t load_bits(const uint16_t* p, int64_t i) { return p[i]; }
template <typename TIn>
__device__ __forceinline__ float bits_value(uint32_t b) {
  if constexpr (sizeof(TIn) == 2) return __uint_as_float(b << 16);
  else return __uint_as_float(b);
}
__device__ __forceinline__ float load_elt(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_elt(const uint16_t* p, int64_t i) { return bf2f(p[i]); }
__device__ __forceinline__ void store_elt(float* p, int64_t i, float x) { p[i] = x; }
__device__ __forceinline__ void store_elt(uint16_t* p, int64_t i, float x) { p[i] = f2bf(x); }

// A-operand fragment in kperm order from an LDS row: elements c0..c0+3 and
// c0+16..c0+19 (two 8-byte reads), c0 = 32 kk + 4 (lane / 16).
__device__ __forceinline__ bf16x8 perm_frag(const uint16_t* p) {
  return join_halves(*reinterpret_cast<const u32x2*>(p), *reinterpret_cast<const u32x2*>(p + 16));
}

// ---------------------------------------------------------------- chunk row tiles
// The 64 chunk rows of one head of a token-major [T, H, D] tensor, held as
// 16-byte vectors spread over a 256-thread workgroup.  `base` points at row 0
// of the head; row i starts `row_stride` elements later.  Rows at or past
// `rows` (1 <= rows <= 64) read as zero: the loads themselves are unconditional
// (clamped to the last valid row) so no load waits behind a branch, and the
// padding is applied when the tile is written to LDS.
template <typename TIn, int D>
struct RowTile {
  static constexpr int kVecPerRow = D * static_cast<int>(sizeof(TIn)) / 16;
  static constexpr int kElemsPerVec = 16 / static_cast<int>(sizeof(TIn));
  static constexpr int kPerThread = 64 * kVecPerRow / 256;
  u32x4 d[kPerThread];
  int rows;

  __device__ __forceinline__ static int row(int tid, int m) { return (tid + 256 * m) / kVecPerRow; }
  __device__ __forceinline__ static int col(int tid, int m) {
    return ((tid + 256 * m) % kVecPerRow) * kElemsPerVec;
  }
  __device__ __forceinline__ void load(const TIn* __restrict__ base, int64_t row_stride, int nrows,
                                       int tid) {
    rows = nrows;
#pragma unroll
    for (int m = 0; m < kPerThread; ++m) {
      const int i = min(row(tid, m), nrows - 1);
      d[m] = *reinterpret_cast<const u32x4*>(base + i * row_stride + col(tid, m));
    }
  }
  __device__ __forceinline__ u32x4 get(int tid, int m) const {
    return row(tid, m) < rows ? d[m] : u32x4{0u, 0u, 0u, 0u};
  }
};

// Element j of a 16-byte vector as float (bf16 or fp32 payload).
template <typename TIn>
__device__ __forceinline__ float vec_elt(const u32x4& u, int j) {
  if constexpr (sizeof(TIn) == 2) {
    const uint32_t w = (j < 2) ? u.x : (j < 4) ? u.y : (j < 6) ? u.z : u.w;
    return __uint_as_float((j & 1) ? (w & 0xFFFF0000u) : (w << 16));
  } else {
    const uint32_t w = (j == 0) ? u.x : (j == 1) ? u.y : (j == 2) ? u.z : u.w;
    return __uint_as_float(w);
  }
}

// Writes a tile row-major into LDS as bf16: dst[p][row][col], p = 0 for the
// value (bf16 input) or the high part, p = 1 for the low part (fp32 input).
template <typename TIn, int D, int NL, int PITCH>
__device__ __forceinline__ void store_rows(uint16_t (*dst)[64][PITCH], const RowTile<TIn, D>& t,
                                           int tid) {
#pragma unroll
  for (int m = 0; m < RowTile<TIn, D>::kPerThread; ++m) {
    const int i = RowTile<TIn, D>::row(tid, m), c = RowTile<TIn, D>::col(tid, m);
    const u32x4 val = t.get(tid, m);
    if constexpr (sizeof(TIn) == 2) {
      *reinterpret_cast<u32x4*>(&dst[0][i][c]) = val;
    } else {
      uint16_t hi[4], lo[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) split_bf16(vec_elt<TIn>(val, j), hi[j], lo[j]);
      *reinterpret_cast<u32x2*>(&dst[0][i][c]) =
          u32x2{hi[0] | (uint32_t(hi[1]) << 16), hi[2] | (uint32_t(hi[3]) << 16)};
      *reinterpret_cast<u32x2*>(&dst[NL - 1][i][c]) =
          u32x2{lo[0] | (uint32_t(lo[1]) << 16), lo[2] | (uint32_t(lo[3]) << 16)};
    }
  }
}

// Writes a tile transposed into LDS as bf16: dst[p][col][row].
template <typename TIn, int D, int NL, int PITCH>
__device__ __forceinline__ void store_cols(uint16_t (*dst)[D][PITCH], const RowTile<TIn, D>& t,
                                           int tid) {
  constexpr int E = RowTile<TIn, D>::kElemsPerVec;
#pragma unroll
  for (int m = 0; m < RowTile<TIn, D>::kPerThread; ++m) {
    const int i = RowTile<TIn, D>::row(tid, m), c = RowTile<TIn, D>::col(tid, m);
    const u32x4 val = t.get(tid, m);
#pragma unroll
    for (int j = 0; j < E; ++j) {
      if constexpr (sizeof(TIn) == 2) {
        const uint32_t w = (j < 2) ? val.x : (j < 4) ? val.y : (j < 6) ? val.z : val.w;
        dst[0][c + j][i] = static_cast<uint16_t>((j & 1) ? (w >> 16) : (w & 0xFFFFu));
      } else {
        uint16_t hi, lo;
        split_bf16(vec_elt<TIn>(val, j), hi, lo);
        dst[0][c + j][i] = hi;
        dst[NL - 1][c + j][i] = lo;
      }
    }
  }
}

}  // namespace gdn
