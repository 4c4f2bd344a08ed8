// Chunk scan kernel: the sequential part of the recurrence.
//
// One workgroup per (sequence, value head): d_v/16 waves (two per SIMD for
// d_v = 128), each owning 16 columns of M = S^T (d_k x d_v) in registers for the
// whole sequence.  Per 64-token chunk, with M0 the state at chunk start:
//   R      = diag(beta) V - diag(beta e^G) (K M0)
//   Delta  = T R                                                  (T from k_intra)
//   O      = diag(scale e^G) (Q M0) + P Delta                     (outputs only)
//   M1     = e^{G_last} M0 + K^T diag(e^{G_last - G}) Delta
// All four products run on MFMA.  The contraction order inside every 32-wide k
// step is permuted (kperm) so each accumulator is directly the next product's
// B operand.  fp32 operands (M0, R, Delta, T, P) are split into bf16 hi + lo.
// For bf16 inputs T R takes two passes, hi(T) (hi + lo)(R); every other
// product keeps both parts of its fp32 operands.  With hi(T) alone the state's
// error stays below about 5e-4 relative (gate scales 0 to 0.5, beta up to 1,
// tails of 3277 tokens and a 32768-token prefix), measured on the CPU with a
// model of exactly these roundings; dropping any other pass (hi(M0) alone in
// K M0, or the lo part of R, Delta or P) takes it past 1e-3 somewhere.
//
// Every A operand except P (K, K^T, Q, T) comes from a workspace record that
// k_intra wrote in fragment order, copied global -> LDS by DMA (global_load_lds,
// 16 bytes per lane) into one of two LDS buffers while the waves compute on the
// other; each wave issues an equal share of the next chunk's DMA at the start
// of a chunk and waits for it at the end.  A wave then fetches each operand
// with one conflict-free 16-byte LDS read; V uses the transposing LDS read; P
// (outputs only) comes straight from global memory into registers.  Two waves
// per SIMD let one wave's VALU work (hi/lo splits) run while the other's MFMAs
// run.  Inside a chunk the waves issue each group of LDS reads one region
// ahead of its use.
#pragma once

#include "gdn_device.h"
#include "gdn_intra.h"
#include "gdn_plan.h"

#include <type_traits>

namespace gdn {

constexpr int kLdsBytes = 160 * 1024;

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef __attribute__((address_space(3))) unsigned char lds_byte;   // LDS bytes

// 16 bytes per lane from `src` (per lane) to LDS `dst + 16 * lane` (dst uniform).
__device__ __forceinline__ void dma16(const void* src, lds_byte* dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)dst, 16, 0, 0);
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// The same from `base + off`: a uniform base and a 32-bit lane offset, so the
// load takes the scalar-base form and its address costs no 64-bit lane
// arithmetic.  Offsets stay below 2^32: a chunk spans 64 rows of at most
// 65535 heads x 128 x 4 bytes.
__device__ __forceinline__ void dma16_at(const void* base, uint32_t off, lds_byte* dst) {
  dma16(static_cast<const unsigned char*>(base) + off, dst);
}


// Byte offset of byte `byte_in_row` of row `row` in a row tile whose rows hold
// ROW_BYTES / 16 pieces of 16 bytes, piece p of row R stored at p ^ (R % pieces).
template <int ROW_BYTES>
__device__ __forceinline__ int swz(int row, int byte_in_row) {
  constexpr int pieces = ROW_BYTES / 16;
  return row * ROW_BYTES + 16 * ((byte_in_row / 16) ^ (row % pieces)) + byte_in_row % 16;
}

// DMA of rows [0, 64) of a token-major tensor (row 0 at `row0`, 1 KiB block
// `blk` of the tile) into a swizzled LDS row tile; rows past `rows` repeat the
// last valid row.
template <int ROW_BYTES, typename T>
__device__ __forceinline__ void dma_rows(const T* row0, int64_t row_stride, int rows, lds_byte* dst,
                                         int blk, int lane) {
  constexpr int pieces = ROW_BYTES / 16;
  constexpr int rows_per_block = 1024 / ROW_BYTES;
  const int r = blk * rows_per_block + lane / pieces;
  const int p = (lane % pieces) ^ (r % pieces);
  const uint32_t stride_b = static_cast<uint32_t>(row_stride) * static_cast<uint32_t>(sizeof(T));
  dma16_at(row0, static_cast<uint32_t>(min(r, rows - 1)) * stride_b + 16u * p, dst + blk * 1024);
}

// Element j (0..3) of four bf16 values packed in two dwords, as float.
__device__ __forceinline__ float bf16_elt(const u32x2& x, int j) {
  const uint32_t w = j < 2 ? x.x : x.y;
  return __uint_as_float((j & 1) ? (w & 0xFFFF0000u) : (w << 16));
}

// Buffer resource over `bytes` bytes from `base` (gfx9 raw buffer: stride 0,
// byte offsets).  The hardware drops a store whose VGPR offset is at or past
// `bytes`; the SGPR offset is not range-checked, so callers pass 0 there.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t out_rsrc(void* base, int bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, 0, bytes, 0x00020000);
}
// Four consecutive output elements of one row, as bf16 (8 bytes) or fp32 (16).
__device__ __forceinline__ void store_out4(__amdgpu_buffer_rsrc_t r, int voff, const f32x4& x, uint16_t*) {
  const uint32_t a = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x[0], x[1]}, bf16x2));
  const uint32_t b = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x[2], x[3]}, bf16x2));
  __builtin_amdgcn_raw_buffer_store_b64(u32x2{a, b}, r, voff, 0, 0);
}
__device__ __forceinline__ void store_out4(__amdgpu_buffer_rsrc_t r, int voff, const f32x4& x, float*) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, x), r, voff, 0, 0);
}

// LDS layout of one chunk buffer of a workgroup that covers VC state columns;
// P (outputs only) is staged in LDS when P_LDS, else read from global memory.
template <typename TIn, int DK, int VC, bool FWD, bool P_LDS>
struct ScanLds {
  static constexpr int kDK = DK;
  static constexpr bool kSplit = sizeof(TIn) == 4;
  static constexpr bool kPInLds = FWD && P_LDS;
  static constexpr int kKFrags = k_record_frags(DK, FWD);         // per bf16 part
  static constexpr int kKBytes = static_cast<int>(k_tile_bytes(DK, FWD, kSplit));
  static constexpr int kTBytes = static_cast<int>(t_record_bytes(kSplit));
  static constexpr int kSBytes = static_cast<int>(kSRecordBytes);
  static constexpr int kVRowBytes = VC * static_cast<int>(sizeof(TIn));
  static constexpr int kVBytes = kChunk * kVRowBytes;
  static constexpr int kOffK = 0;                 // K (and Q) fragments
  static constexpr int kOffT = kOffK + kKBytes;
  static constexpr int kPBytes = kPInLds ? static_cast<int>(kPRecordBytes) : 0;
  static constexpr int kOffP = kOffT + kTBytes;
  static constexpr int kOffS = kOffP + kPBytes;
  static constexpr int kOffV = kOffS + 2048;      // S padded to two DMA blocks
  static constexpr int kBytes = kOffV + kVBytes;
  static constexpr int kBuffers = 2 * kBytes <= kLdsBytes ? 2 : 1;
  // DMA jobs per chunk (one 1 KiB global_load_lds each): K (and Q) fragments,
  // T, P, V rows, then the scalars as one full and one quarter block
  static constexpr int kKJobs = kKBytes / 1024, kTJobs = kTBytes / 1024, kPJobs = kPBytes / 1024;
  static constexpr int kVJobs = kVBytes / 1024;
  static constexpr int kJobs = kKJobs + kTJobs + kPJobs + kVJobs + 2;
};

// Where one chunk's operands come from.
struct ChunkSrc {
  const unsigned char* krec;   // K record of (slot, key head), fp32 inputs
  const void* k0;              // key row 0 of the chunk (bf16 inputs: the fragments come from the rows)
  const void* q0;              // query row 0 of the chunk (bf16 inputs, outputs only)
  int64_t krow;                // elements between consecutive key (query) rows
  const unsigned char* trec;   // T record of (slot, value head)
  const unsigned char* prec;   // P record of (slot, value head), outputs only
  const unsigned char* srow;   // scalars of (slot, value head)
  const void* v0;              // V row 0 of the chunk, first column of the workgroup
  int clen;                    // valid rows
};

// DMA job j of a chunk (0 <= j < L::kJobs) into LDS buffer `base`.
template <typename L, typename TIn>
__device__ __forceinline__ void dma_job(const ChunkSrc& c, int64_t vrow, lds_byte* base, int j, int lane) {
  if (j < L::kKJobs) {
    if constexpr (L::kSplit) {
      dma16_at(c.krec + 1024 * j, 16u * lane, base + L::kOffK + 1024 * j);
    } else {
      // fragment j: keys for j < 4 d_k/32, then queries; the lane at position
      // `lane` (kslot order) takes 16 bytes of row 16 ti + r at column 32 kk +
      // 8 g; pad rows repeat the last row (their beta is 0, so they add nothing)
      constexpr int NK = L::kDK / 32, NKA = ka_frags(L::kDK);
      const bool isq = j >= NKA;
      const int f = isq ? j - NKA : j;
      const int l = kslot_inv(lane);
      const int row = min(16 * (f / NK) + (l & 15), c.clen - 1);
      const uint32_t krow_b = static_cast<uint32_t>(c.krow) * 2u;
      dma16_at(static_cast<const uint16_t*>(isq ? c.q0 : c.k0) + 32 * (f % NK),
               static_cast<uint32_t>(row) * krow_b + 16u * (l >> 4), base + L::kOffK + 1024 * j);
    }
  } else if (j < L::kKJobs + L::kTJobs) {
    const int t = j - L::kKJobs;
    dma16_at(c.trec + 1024 * t, 16u * lane, base + L::kOffT + 1024 * t);
  } else if (j < L::kKJobs + L::kTJobs + L::kPJobs) {
    const int t = j - L::kKJobs - L::kTJobs;
    dma16_at(c.prec + 1024 * t, 16u * lane, base + L::kOffP + 1024 * t);
  } else if (j < L::kKJobs + L::kTJobs + L::kPJobs + L::kVJobs) {
    // V rows; pad rows repeat the last row (their beta is 0, so they add nothing)
    dma_rows<L::kVRowBytes>(static_cast<const TIn*>(c.v0), vrow, c.clen, base + L::kOffV,
                            j - L::kKJobs - L::kTJobs - L::kPJobs, lane);
  } else if (j == L::kJobs - 2) {
    dma16_at(c.srow, 16u * lane, base + L::kOffS);                 // scalars, bytes 0..1023
  } else if (lane < 16) {
    dma16_at(c.srow + 1024, 16u * lane, base + L::kOffS + 1024);   // bytes 1024..1279
  }
}

// One 64-token chunk for one wave: 16 state columns, M (and its split mb) in
// registers.  `base` is the chunk's LDS buffer, `vc0` the wave's first column
// within the buffer's V tile, `pg` the chunk's P record in global memory
// (outputs only, used when the layout does not stage P in LDS).  The chunk runs as a chain of regions: each region issues the
// LDS reads of a later region, runs MFMAs on operands that are ready, and does
// VALU work (scaling, hi/lo splits) for the next region that is independent of
// its own MFMAs.  hook(k) runs at the start of region k (the whole-head kernel
// issues its DMA share there).  With outputs, the chunk's O is left in `pout`:
// pout[ti][i] = O[16 ti + lane % 16][4 (lane / 16) + i] of the wave's columns.
// With EXPORT (and FWD false), the wave leaves the outputs to another wave: it
// writes Delta (four 16-byte tiles per lane) to LDS `xd` before hook(5) and
// the split of M1 (the next chunk's B operand of K M0, layout [k step][hi |
// lo][lane]) to `xm` at the end.
template <typename L, int DK, bool FWD, bool EXPORT, typename Hook>
__device__ __forceinline__ void chunk_step(const unsigned char* base, int vc0, const u32x4* pg, int lane,
                                           f32x4 (&M)[DK / 16], Frag (&mb)[DK / 32], f32x4 (&pout)[4],
                                           Hook&& hook, unsigned char* xd = nullptr,
                                           unsigned char* xm = nullptr) {
  static_assert(!(FWD && EXPORT), "a wave that exports Delta leaves the outputs to another");
  constexpr bool SPLIT = L::kSplit;
  constexpr int NT = DK / 16, NK = DK / 32;
  constexpr int NKA = ka_frags(DK);
  constexpr int NKF = L::kKFrags;
  constexpr int VRB = L::kVRowBytes;
  const int lg = lane / 16, lr = lane % 16;
  const u32x4* kf = reinterpret_cast<const u32x4*>(base + L::kOffK);
  const u32x4* tf = reinterpret_cast<const u32x4*>(base + L::kOffT);
  const float* sc = reinterpret_cast<const float*>(base + L::kOffS);
  const unsigned char* vtile = base + L::kOffV;
  // fragment f of the K record (`nf` fragments per bf16 part; the lo part
  // exists for fp32 inputs only), lanes in kslot order
  const int klane = kslot(lane);
  auto ldf = [&](Frag& x, const u32x4* rec, int f, int nf) __attribute__((always_inline)) {
    x.hi = __builtin_bit_cast(bf16x8, rec[f * kWave + klane]);
    if constexpr (SPLIT) x.lo = __builtin_bit_cast(bf16x8, rec[(nf + f) * kWave + klane]);
  };
  // fp32-derived records: P always hi and lo, T hi (and lo for fp32 inputs)
  auto ld_split = [&](Frag& x, const u32x4* rec, int f) __attribute__((always_inline)) {
    x.hi = __builtin_bit_cast(bf16x8, rec[f * kWave + lane]);
    x.lo = __builtin_bit_cast(bf16x8, rec[(kTFrags + f) * kWave + lane]);
  };
  auto ld_t = [&](Frag& x, const u32x4* rec, int f) __attribute__((always_inline)) {
    x.hi = __builtin_bit_cast(bf16x8, rec[f * kWave + lane]);
    if constexpr (SPLIT) x.lo = __builtin_bit_cast(bf16x8, rec[(kTFrags + f) * kWave + lane]);
  };
  // K M0: K exact (bf16 inputs) or split (fp32 inputs), M0 split
  auto mma_km = [&](const Frag& a, const Frag& m, f32x4 c) __attribute__((always_inline)) {
    return mma_a<SPLIT>(a, m, c);
  };
  // T R: fp32 inputs 3 passes; bf16 inputs hi(T) times both parts of R
  auto mma_tr = [&](const Frag& t, const Frag& r, f32x4 c) __attribute__((always_inline)) {
    if constexpr (SPLIT) return mma_x3(t, r, c);
    else return mma_x2(t.hi, r, c);
  };
  // K (and Q) operands of row tiles 2 tp, 2 tp + 1 for every k step
  auto ld_ka = [&](Frag (&a)[2][NK], Frag (&aq)[2][NK], int tp) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        ldf(a[u][kk], kf, (2 * tp + u) * NK + kk, NKF);
        if constexpr (FWD) ldf(aq[u][kk], kf, NKA + (2 * tp + u) * NK + kk, NKF);
      }
  };
  // K^T operands of every row tile td of M for token k step kk, by
  // transposing reads of the K fragments: lane (g, c) needs K[32 kk +
  // kperm(g, j)][16 td + c].  In a transposing read each lane of a 16-lane
  // group addresses four consecutive columns of one row and receives one
  // column of four rows; lane (g, c) addresses row 32 kk + 4 g + c / 4
  // (then 16 rows further, for j >= 4), columns 16 td + 4 (c % 4)..+3: in K
  // fragment (row tile 2 kk (+1), k step td / 2) that is lane 16 (c % 4) +
  // 4 g + c / 4 (at its kslot position), bytes 8 (td % 2)..+7.
  const int kt_off = 16 * kslot(16 * (lr % 4) + 4 * lg + lr / 4);
  auto ld_kt = [&](Frag (&a)[NT], int kk) __attribute__((always_inline)) {
#pragma unroll
    for (int td = 0; td < NT; ++td) {
      const unsigned char* f0 = reinterpret_cast<const unsigned char*>(kf + ((2 * kk) * NK + td / 2) * kWave);
      const unsigned char* f1 = reinterpret_cast<const unsigned char*>(kf + ((2 * kk + 1) * NK + td / 2) * kWave);
      const int o = kt_off + 8 * (td % 2);
      a[td].hi = __builtin_bit_cast(bf16x8, join_halves(lds_read_tr16(f0 + o), lds_read_tr16(f1 + o)));
      if constexpr (SPLIT) {
        constexpr int lo = NKF * kWave * 16;
        a[td].lo = __builtin_bit_cast(bf16x8, join_halves(lds_read_tr16(f0 + lo + o), lds_read_tr16(f1 + lo + o)));
      }
    }
  };

  // The chunk runs as a chain of regions.  Each region issues the LDS reads of
  // a later region, runs MFMAs on operands that are ready, and does VALU work
  // (scaling, hi/lo splits) for the next region, independent of its own MFMAs
  // so the two overlap.
  Frag ka0[2][NK], qa0[2][NK], ka1[2][NK], qa1[2][NK];
  Frag tfr[kTFrags];
  Frag kt0[NT], kt1[NT];
  f32x4 km[4], qm[4], bv[4], R[4], D[4];
  u32x2 vraw[4];
  float vf[4][4];

  hook(0);
  // ---- region 0: first operands
  ld_ka(ka0, qa0, 0);
  if constexpr (!SPLIT) {
    // transposing read: lane (g, c) gets V[16 ti + 4 g + r][c], r = 0..3
#pragma unroll
    for (int ti = 0; ti < 4; ++ti)
      vraw[ti] = lds_read_tr16(vtile + swz<VRB>(16 * ti + 4 * lg + lr / 4, 2 * (vc0 + 4 * (lr % 4))));
  } else {
#pragma unroll
    for (int ti = 0; ti < 4; ++ti)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        vf[ti][r] = *reinterpret_cast<const float*>(vtile + swz<VRB>(16 * ti + 4 * lg + r, 4 * (vc0 + lr)));
  }
  __builtin_amdgcn_sched_barrier(0);

  hook(1);
  // ---- region 1: K M0 for row tiles 0, 1 | beta V; the row tiles 2, 3
  //      operands arrive
  ld_ka(ka1, qa1, 1);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    km[u] = zero4();
    qm[u] = zero4();
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      km[u] = mma_km(ka0[u][kk], mb[kk], km[u]);
      if constexpr (FWD) qm[u] = mma_b<SPLIT>(mb[kk], qa0[u][kk], qm[u]);
    }
  }
#pragma unroll
  for (int ti = 0; ti < 4; ++ti) {
    const f32x4 bta = *reinterpret_cast<const f32x4*>(sc + 0 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
    for (int r = 0; r < 4; ++r) bv[ti][r] = bta[r] * (SPLIT ? vf[ti][r] : bf16_elt(vraw[ti], r));
  }
  __builtin_amdgcn_sched_barrier(0);

  hook(2);
  // ---- region 2: K M0 for row tiles 2, 3 | R rows 0..31 and their split;
  //      T arrives
#pragma unroll
  for (int f = 0; f < kTFrags; ++f) ld_t(tfr[f], tf, f);
#pragma unroll
  for (int u = 0; u < 2; ++u) {
    km[2 + u] = zero4();
    qm[2 + u] = zero4();
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      km[2 + u] = mma_km(ka1[u][kk], mb[kk], km[2 + u]);
      if constexpr (FWD) qm[2 + u] = mma_b<SPLIT>(mb[kk], qa1[u][kk], qm[2 + u]);
    }
  }
  auto make_r = [&](int ti) __attribute__((always_inline)) {
    const f32x4 bge = *reinterpret_cast<const f32x4*>(sc + 1 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
    for (int r = 0; r < 4; ++r) R[ti][r] = bv[ti][r] - bge[r] * km[ti][r];
  };
  make_r(0);
  make_r(1);
  const Frag rb0 = chain_frag(R[0], R[1]);
  __builtin_amdgcn_sched_barrier(0);

  hook(3);
  // ---- region 3: Delta = T R, k step 0 for all row tiles | R rows 32..63
  //      and their split; K^T (k step 0) and P (outputs) arrive
  ld_kt(kt0, 0);
  Frag pfr[FWD ? kTFrags : 1];
  if constexpr (FWD) {
    // P (fp32-derived: hi and lo parts), staged in LDS or straight from global
    if constexpr (L::kPInLds) {
      const u32x4* pl = reinterpret_cast<const u32x4*>(base + L::kOffP);
#pragma unroll
      for (int f = 0; f < kTFrags; ++f) ld_split(pfr[f], pl, f);
    } else {
#pragma unroll
      for (int f = 0; f < kTFrags; ++f) {
        pfr[f].hi = __builtin_bit_cast(bf16x8, pg[f * kWave + lane]);
        pfr[f].lo = __builtin_bit_cast(bf16x8, pg[(kTFrags + f) * kWave + lane]);
      }
    }
  }
#pragma unroll
  for (int ti = 0; ti < 4; ++ti) D[ti] = mma_tr(tfr[tri_frag(ti, 0)], rb0, zero4());
  make_r(2);
  make_r(3);
  const Frag rb1 = chain_frag(R[2], R[3]);
  __builtin_amdgcn_sched_barrier(0);

  hook(4);
  // ---- region 4: Delta, k step 1 for row tiles 2, 3 | split of the
  //      weighted Delta rows 0..31 (and of Delta for the outputs); K^T
  //      arrives
  ld_kt(kt1, 1);
  if constexpr (EXPORT) {
#pragma unroll
    for (int ti = 0; ti < 2; ++ti) reinterpret_cast<f32x4*>(xd)[ti * kWave + lane] = D[ti];   // final
  }
#pragma unroll
  for (int ti = 2; ti < 4; ++ti) D[ti] = mma_tr(tfr[tri_frag(ti, 1)], rb1, D[ti]);
  f32x4 Dw[4];
  auto make_dw = [&](int ti) __attribute__((always_inline)) {
    const f32x4 w = *reinterpret_cast<const f32x4*>(sc + 2 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
    for (int r = 0; r < 4; ++r) Dw[ti][r] = w[r] * D[ti][r];
  };
  make_dw(0);
  make_dw(1);
  const Frag db0 = chain_frag(Dw[0], Dw[1]);
  Frag dd0;
  if constexpr (FWD) dd0 = chain_frag(D[0], D[1]);
  __builtin_amdgcn_sched_barrier(0);

  if constexpr (EXPORT) {
#pragma unroll
    for (int ti = 2; ti < 4; ++ti) reinterpret_cast<f32x4*>(xd)[ti * kWave + lane] = D[ti];
  }
  hook(5);
  // ---- region 5: M1 partial, k step 0 (tokens 0..31) | split of the
  //      weighted Delta rows 32..63
  const float eg = sc[4 * kChunk];
#pragma unroll
  for (int td = 0; td < NT; ++td) {
#pragma unroll
    for (int r = 0; r < 4; ++r) M[td][r] *= eg;
    M[td] = mma_a<SPLIT>(kt0[td], db0, M[td]);
  }
  make_dw(2);
  make_dw(3);
  const Frag db1 = chain_frag(Dw[2], Dw[3]);
  Frag dd1;
  if constexpr (FWD) dd1 = chain_frag(D[2], D[3]);
  __builtin_amdgcn_sched_barrier(0);

  // ---- outputs, transposed: O^T = diag-scaled (Q M0)^T + Delta^T P^T, whose
  //      MFMA layout gives a lane four consecutive columns of one token row
  //      (row 16 ti + lane % 16, columns 4 (lane / 16) + 0..3 of the wave's 16).
  //      The split Delta (dd) is the A operand and the P fragments the B
  //      operand; qm already holds (Q M0)^T (A = split M0, B = Q fragments).
  //      Stored at the start of the next chunk.
  if constexpr (FWD) {
#pragma unroll
    for (int ti = 0; ti < 4; ++ti) {
      const float qe = sc[3 * kChunk + 16 * ti + lr];
#pragma unroll
      for (int r = 0; r < 4; ++r) pout[ti][r] = qe * qm[ti][r];
      pout[ti] = mma_x3(dd0, pfr[tri_frag(ti, 0)], pout[ti]);
      if (ti >= 2) pout[ti] = mma_x3(dd1, pfr[tri_frag(ti, 1)], pout[ti]);
    }
    __builtin_amdgcn_sched_barrier(0);
  }

  hook(6);
  // ---- region 6: M1, k step 1 (tokens 32..63) | split of M1 for the next chunk
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) {
    M[2 * kk] = mma_a<SPLIT>(kt1[2 * kk], db1, M[2 * kk]);
    M[2 * kk + 1] = mma_a<SPLIT>(kt1[2 * kk + 1], db1, M[2 * kk + 1]);
    mb[kk] = chain_frag(M[2 * kk], M[2 * kk + 1]);
  }
  if constexpr (EXPORT) {
    u32x4* x = reinterpret_cast<u32x4*>(xm);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      x[(2 * kk) * kWave + lane] = __builtin_bit_cast(u32x4, mb[kk].hi);
      x[(2 * kk + 1) * kWave + lane] = __builtin_bit_cast(u32x4, mb[kk].lo);
    }
  }
}

// One 64-token chunk of tail replay (no outputs, bf16 inputs) for a wave that
// carries NC tiles of 16 state columns: the products of chunk_step in the same
// order with the same roundings (so the state is bit for bit that of NC waves
// of one tile each), but every operand that does not depend on the state (K,
// T, K^T) is read from LDS once for all NC tiles, and K M0 runs k step by k
// step (the four row tiles' K fragments of one step, shared by the tiles), so
// only two steps' operands are held at a time.  The tiles' chains are
// independent, so each phase has NC times the MFMAs to cover the LDS reads
// issued for the next.  hook(p) runs at the start of phase p, p = 0 ..
// tiles_phases(DK) - 1 (a workgroup without a DMA wave issues the next
// chunk's DMA there).
constexpr int tiles_phases(int dk) { return dk / 32 + 6; }
template <typename L, int DK, int NC, typename Hook>
__device__ __forceinline__ void chunk_step_tiles(const unsigned char* base, int vc0, int lane,
                                                 f32x4 (&M)[NC][DK / 16], Frag (&mb)[NC][DK / 32],
                                                 Hook&& hook) {
  static_assert(!L::kSplit, "bf16 inputs: K, K^T and hi(T) are single bf16 operands");
  constexpr int NT = DK / 16, NK = DK / 32;
  constexpr int VRB = L::kVRowBytes;
  const int lg = lane / 16, lr = lane % 16;
  const u32x4* kf = reinterpret_cast<const u32x4*>(base + L::kOffK);
  const u32x4* tf = reinterpret_cast<const u32x4*>(base + L::kOffT);
  const float* sc = reinterpret_cast<const float*>(base + L::kOffS);
  const unsigned char* vtile = base + L::kOffV;
  const int klane = kslot(lane);
  // K fragment of row tile ti, k step kk (lanes in kslot order)
  auto ldk = [&](int ti, int kk) __attribute__((always_inline)) {
    return __builtin_bit_cast(bf16x8, kf[(ti * NK + kk) * kWave + klane]);
  };
  // K^T operand of row tile td of M for token k step kk (as in chunk_step)
  const int kt_off = 16 * kslot(16 * (lr % 4) + 4 * lg + lr / 4);
  auto ldkt = [&](int td, int kk) __attribute__((always_inline)) {
    const unsigned char* f0 = reinterpret_cast<const unsigned char*>(kf + ((2 * kk) * NK + td / 2) * kWave);
    const unsigned char* f1 = reinterpret_cast<const unsigned char*>(kf + ((2 * kk + 1) * NK + td / 2) * kWave);
    const int o = kt_off + 8 * (td % 2);
    return __builtin_bit_cast(bf16x8, join_halves(lds_read_tr16(f0 + o), lds_read_tr16(f1 + o)));
  };

  // ---- V (transposing reads: lane (g, c) gets V[16 ti + 4 g + r][c]) and the
  //      first k step's K
  hook(0);
  u32x2 vraw[NC][4];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int ti = 0; ti < 4; ++ti)
      vraw[c][ti] = lds_read_tr16(vtile + swz<VRB>(16 * ti + 4 * lg + lr / 4, 2 * (vc0 + 16 * c + 4 * (lr % 4))));
  bf16x8 ka[2][4];
#pragma unroll
  for (int ti = 0; ti < 4; ++ti) ka[0][ti] = ldk(ti, 0);
  __builtin_amdgcn_sched_barrier(0);

  // ---- K M0, one k step at a time; the next step's K (after the last, T) arrives
  f32x4 km[NC][4];
  bf16x8 tfr[kTFrags];
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) {
    hook(1 + kk);
    if (kk + 1 < NK) {
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) ka[(kk + 1) & 1][ti] = ldk(ti, kk + 1);
    } else {
#pragma unroll
      for (int f = 0; f < kTFrags; ++f) tfr[f] = __builtin_bit_cast(bf16x8, tf[f * kWave + lane]);
    }
#pragma unroll
    for (int ti = 0; ti < 4; ++ti)
#pragma unroll
      for (int c = 0; c < NC; ++c)
        km[c][ti] = mma_x2(ka[kk & 1][ti], mb[c][kk], kk == 0 ? zero4() : km[c][ti]);
    __builtin_amdgcn_sched_barrier(0);
  }

  // ---- R = diag(beta) V - diag(beta e^G) (K M0), split by 32-row halves
  hook(NK + 1);
  bf16x8 kt0[NT], kt1[NT];
  Frag rb[NC][2];
  auto make_rb = [&](int h) __attribute__((always_inline)) {
    f32x4 R[NC][2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int ti = 2 * h + u;
      const f32x4 bta = *reinterpret_cast<const f32x4*>(sc + 0 * kChunk + 16 * ti + 4 * lg);
      const f32x4 bge = *reinterpret_cast<const f32x4*>(sc + 1 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) R[c][u][r] = bta[r] * bf16_elt(vraw[c][ti], r) - bge[r] * km[c][ti][r];
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) rb[c][h] = chain_frag(R[c][0], R[c][1]);
  };
  make_rb(0);
  __builtin_amdgcn_sched_barrier(0);

  // ---- Delta = hi(T) R, k step 0 | R rows 32..63; K^T for tokens 0..31 arrives
  hook(NK + 2);
#pragma unroll
  for (int td = 0; td < NT; ++td) kt0[td] = ldkt(td, 0);
  f32x4 D[NC][4];
#pragma unroll
  for (int ti = 0; ti < 4; ++ti)
#pragma unroll
    for (int c = 0; c < NC; ++c) D[c][ti] = mma_x2(tfr[tri_frag(ti, 0)], rb[c][0], zero4());
  make_rb(1);
  __builtin_amdgcn_sched_barrier(0);

  // ---- Delta, k step 1 for row tiles 2, 3 | the weighted Delta rows 0..31,
  //      split; K^T for tokens 32..63 arrives
  hook(NK + 3);
#pragma unroll
  for (int td = 0; td < NT; ++td) kt1[td] = ldkt(td, 1);
#pragma unroll
  for (int ti = 2; ti < 4; ++ti)
#pragma unroll
    for (int c = 0; c < NC; ++c) D[c][ti] = mma_x2(tfr[tri_frag(ti, 1)], rb[c][1], D[c][ti]);
  Frag db[NC][2];
  auto make_db = [&](int h) __attribute__((always_inline)) {
    f32x4 Dw[NC][2];
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const f32x4 w = *reinterpret_cast<const f32x4*>(sc + 2 * kChunk + 16 * (2 * h + u) + 4 * lg);
#pragma unroll
      for (int c = 0; c < NC; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) Dw[c][u][r] = w[r] * D[c][2 * h + u][r];
    }
#pragma unroll
    for (int c = 0; c < NC; ++c) db[c][h] = chain_frag(Dw[c][0], Dw[c][1]);
  };
  make_db(0);
  const float eg = sc[4 * kChunk];
  __builtin_amdgcn_sched_barrier(0);

  // ---- M1 = e^{G_last} M0 + K^T Dw, tokens 0..31 | weighted Delta rows 32..63
  hook(NK + 4);
#pragma unroll
  for (int td = 0; td < NT; ++td)
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int r = 0; r < 4; ++r) M[c][td][r] *= eg;
      M[c][td] = mma_x2(kt0[td], db[c][0], M[c][td]);
    }
  make_db(1);
  __builtin_amdgcn_sched_barrier(0);

  // ---- tokens 32..63 | split of M1 for the next chunk
  hook(NK + 5);
#pragma unroll
  for (int kk = 0; kk < NK; ++kk)
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      M[c][2 * kk] = mma_x2(kt1[2 * kk], db[c][1], M[c][2 * kk]);
      M[c][2 * kk + 1] = mma_x2(kt1[2 * kk + 1], db[c][1], M[c][2 * kk + 1]);
      mb[c][kk] = chain_frag(M[c][2 * kk], M[c][2 * kk + 1]);
    }
}

// Shared set-up of a scan workgroup for sequence n, value head h, state
// columns [col0, col0 + VC).
struct ScanUnit {
  int n, h, kh, tok0, len, slot0, nch;
};
// `slot` is the workgroup's logical sequence slot; `order` (NULL or n = 0:
// identity) maps it to the sequence, longest first.  When a scan grid exceeds
// the chip, workgroups start in logical order as earlier ones finish, so a
// long sequence that comes late in a varlen batch would finish late.
__device__ __forceinline__ ScanUnit scan_unit(const int32_t* __restrict__ cu, int slot, int h, int hv, int hk,
                                              const SeqOrder* order = nullptr) {
  const int n = (order && order->n > 0) ? order->seq[slot] : slot;
  ScanUnit u;
  u.n = n;
  u.h = h;
  u.kh = h / (hv / hk);
  u.tok0 = cu[n];
  u.len = cu[n + 1] - u.tok0;
  u.slot0 = u.tok0 / kChunk + n;
  u.nch = (u.len + kChunk - 1) / kChunk;
  return u;
}

template <typename L, typename TIn>
__device__ __forceinline__ ChunkSrc chunk_src(const ScanUnit& u, int ci, int hk, int hv, int dv, int col0,
                                              const TIn* v, const TIn* kin, const TIn* qin, const u32x4* Kw,
                                              const u32x4* Tw, const float* Sw, const u32x4* Pw) {
  const int64_t srec = static_cast<int64_t>(u.slot0 + ci);
  const int64_t vrow = static_cast<int64_t>(hv) * dv;
  ChunkSrc c;
  c.krec = reinterpret_cast<const unsigned char*>(Kw) + (srec * hk + u.kh) * L::kKBytes;
  c.krow = static_cast<int64_t>(hk) * L::kDK;
  const int64_t krow0 = static_cast<int64_t>(u.tok0 + ci * kChunk) * c.krow + static_cast<int64_t>(u.kh) * L::kDK;
  c.k0 = kin + krow0;
  c.q0 = qin ? qin + krow0 : nullptr;
  c.trec = reinterpret_cast<const unsigned char*>(Tw) + (srec * hv + u.h) * L::kTBytes;
  c.prec = reinterpret_cast<const unsigned char*>(Pw) + (srec * hv + u.h) * static_cast<int64_t>(kPRecordBytes);
  c.srow = reinterpret_cast<const unsigned char*>(Sw) + (srec * hv + u.h) * L::kSBytes;
  c.v0 = v + static_cast<int64_t>(u.tok0 + ci * kChunk) * vrow + static_cast<int64_t>(u.h) * dv + col0;
  c.clen = min(kChunk, u.len - ci * kChunk);
  return c;
}

// Per-wave state load/store and the deferred output store.
template <int DK>
__device__ __forceinline__ void load_state(const float* __restrict__ state_in, int64_t sbase, int dv, int lg,
                                           f32x4 (&M)[DK / 16], Frag (&mb)[DK / 32]) {
#pragma unroll
  for (int td = 0; td < DK / 16; ++td)
#pragma unroll
    for (int r = 0; r < 4; ++r)
      M[td][r] = state_in ? state_in[sbase + static_cast<int64_t>(strow(td, lg, r)) * dv] : 0.f;
#pragma unroll
  for (int kk = 0; kk < DK / 32; ++kk) mb[kk] = chain_frag(M[2 * kk], M[2 * kk + 1]);
}
// Stores a chunk's outputs (`pout` as chunk_step leaves it) for the wave whose
// first column is `colw`; rows past the chunk's end fall outside the buffer
// range and are dropped by the hardware.
template <typename TIn>
__device__ __forceinline__ void store_chunk_out(TIn* o, const ScanUnit& u, int ci, int hv, int dv, int colw,
                                                int lane, const f32x4 (&pout)[4]) {
  constexpr int E = static_cast<int>(sizeof(TIn));
  const int64_t vrow = static_cast<int64_t>(hv) * dv;
  const int row_bytes = static_cast<int>(vrow) * E;
  const int clen = min(kChunk, u.len - ci * kChunk);
  const __amdgpu_buffer_rsrc_t r =
      out_rsrc(o + static_cast<int64_t>(u.tok0 + ci * kChunk) * vrow + static_cast<int64_t>(u.h) * dv,
               clen * row_bytes);
  const int voff = (lane % 16) * row_bytes + (colw + 4 * (lane / 16)) * E;
#pragma unroll
  for (int ti = 0; ti < 4; ++ti) store_out4(r, voff + 16 * ti * row_bytes, pout[ti], o);
}

// ---------------------------------------------------------------- latency kernel
// grid = N x Hv x d_v/32, one workgroup per CU.  Used when this grid fits on
// the chip at once, where per-chunk latency is all that matters.  Tail replay:
// two compute waves (16 columns each) and one wave that only issues DMA.  With
// outputs: the two waves that carry the recurrence hand Delta and the split
// state to two output waves (one per 16 columns), so the outputs' products
// stay off the sequential chain, and a fifth wave issues the DMA.
constexpr int kColsPerGroup = 32;
// With outputs, bf16 inputs get a dedicated DMA wave; for fp32 inputs the
// recurrence wave needs ~250 VGPRs, more than two waves sharing a SIMD may
// hold, so the two output waves issue the DMA instead (4 waves).
constexpr bool cols_dma_wave(bool fwd, bool split) { return fwd && !split; }
constexpr int cols_threads(bool fwd, bool split, int tiles = 2) {
  return (fwd ? (split ? 4 : 1 + 2 * tiles) : 3) * kWave;
}

template <typename TIn, int DK, bool FWD, int COLS = kColsPerGroup>
using ColsLds = ScanLds<TIn, DK, COLS, FWD, true>;

// Tail replay of bf16 inputs whose grid does not fit on the chip at once (a
// throughput batch) runs the wide column scan: COLS = 128 columns (a whole
// head; 64 for d_v = 64) per workgroup, two 16-column tiles per compute wave
// (chunk_step_tiles: the K, T and K^T operands are read from LDS once for both
// tiles), no DMA wave (each compute wave issues a share of the next chunk's
// DMA), and two workgroups per CU, so every SIMD holds two waves whose chains
// interleave.  Measured on MI355X (16 sequences x 32 heads x 52 chunks):
// 1.25x the columns per CU per unit time of the 64-column workgroup of four
// one-tile waves and a DMA wave it replaces.
constexpr int kWideTiles = 2;   // 16-column tiles per compute wave
constexpr int cols_wide_threads(int cols) { return cols / (16 * kWideTiles) * kWave; }

// Tail replay in two halves: the recurrence over a chunk is affine in the
// state, M1 = A_c M0 + B_c with A_c = e^{G_last} I - K^T diag(e^{G_last - G}) T
// diag(beta e^G) K (d_k x d_k), so the state after chunks [0, n) from zero is
// A M' + M'' where M' is the state after the first c1 chunks, M'' the state
// after the remaining chunks started from zero, and A the product of their
// A_c: the same recurrence run with V = 0 from M0 = I.  The parts run side by
// side in one launch (k_scan_cols_split):
//   first half  (kFirstHalf):  chunks [0, c1), zero start, state -> state_out
//   second half (kSecondHalf): chunks [c1, n), zero start, state -> m2, and
//                              identity start with V = 0, d_k columns -> a2
// and k_state_combine forms A M' + M'' in state_out.  Each part is the
// unsplit scan's arithmetic on its chunks.  The first half runs 32 columns
// per workgroup, the second 64 (four waves read the chunk's operands from LDS,
// and the part starts later), so the first half takes the first
// round(0.54 n) chunks: on MI355X at n = 52 and 26 the halves then end
// closest together (28 of 52: the split scan 47.0 -> 46.3 us against 29).
enum ScanPart { kWhole = 0, kFirstHalf = 1, kSecondHalf = 2 };
struct SplitOut {
  float* m2;   // [N, Hv, d_k, d_v] second half from zero
  float* a2;   // [N, Hv, d_k, d_k] second half's transition, transposed (A^T)
};
__device__ __forceinline__ int split_point(int nch) { return (27 * nch + 25) / 50; }

// One column-split workgroup (block `block` of `nblocks`), LDS in `lds`, COLS
// columns per workgroup, NC tiles of 16 columns per compute wave.  Waves 0 ..
// COLS / (16 NC) - 1 compute.  With DMA_WAVE the next issues the DMA and any
// further waves only take part in the barriers; without, the compute waves
// issue the next chunk's DMA themselves, a share at each phase of the chunk
// (multi-tile steps only).
template <typename TIn, int DK, bool FWD, int COLS = kColsPerGroup, int PART = kWhole, int NC = 1,
          bool DMA_WAVE = true>
__device__ __forceinline__ void scan_cols_body(lds_byte* lds_l, int block, int nblocks,
                                               const int32_t* __restrict__ cu, int32_t hk, int32_t hv,
                                               int32_t dv, const TIn* __restrict__ v,
                                               const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                                               const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                                               const float* __restrict__ Sw, const u32x4* __restrict__ Pw,
                                               const float* __restrict__ state_in, TIn* __restrict__ o,
                                               float* __restrict__ state_out, SplitOut split = {},
                                               const SeqOrder* order = nullptr) {
  using L = ColsLds<TIn, DK, FWD, COLS>;
  constexpr bool SPLIT = PART != kWhole;
  static_assert(!(SPLIT && FWD), "the split form is tail replay only");
  constexpr int NT = DK / 16;
  constexpr int CW = COLS / (16 * NC);   // compute waves
  static_assert(CW * 16 * NC == COLS, "whole column tiles per wave");
  static_assert(DMA_WAVE || NC > 1, "the compute waves issue the DMA in multi-tile steps");
  constexpr int kVJob0 = L::kKJobs + L::kTJobs + L::kPJobs;   // first V job
  const int tid = threadIdx.x;
  // wave index made provably uniform: DMA destinations (M0) stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const bool data_wave = DMA_WAVE && wave >= CW;
  const bool dma_wave = DMA_WAVE && wave == CW;
  const int lane = tid % kWave, lg = lane / 16, lr = lane % 16;
  const int ngroups = PART == kSecondHalf ? dv / COLS + DK / COLS : dv / COLS;
  // logical unit: the column groups of a value head, then the value heads of a
  // key head, are adjacent and one cluster (same XCD, shared records in its L2)
  const int unit = xcd_cluster_remap(block, nblocks, ngroups * (hv / hk));
  const ScanUnit u = scan_unit(cu, unit / (ngroups * hv), (unit / ngroups) % hv, hv, hk, order);
  // this workgroup's chunks [cb, ce), columns, start and destination
  int g = unit % ngroups, cb = 0, ce = u.nch, ld = dv;
  bool ident = false;
  float* dst = state_out;
  if constexpr (PART == kFirstHalf) {
    ce = split_point(u.nch);
  } else if constexpr (PART == kSecondHalf) {
    cb = split_point(u.nch);
    if (g < dv / COLS) {
      dst = split.m2;
    } else {
      g -= dv / COLS;
      ident = true;
      ld = DK;
      dst = split.a2;
    }
  }
  const int col0 = COLS * g;
  const int colw = col0 + 16 * NC * wave;   // the wave's first column; tile c: colw + 16 c + lr
  const int64_t vrow = static_cast<int64_t>(hv) * dv;
  auto dma_chunk = [&](int ci, int b) __attribute__((always_inline)) {
    const ChunkSrc c = chunk_src<L>(u, ci, hk, hv, dv, ident ? 0 : col0, v, kin, qin, Kw, Tw, Sw, Pw);
#pragma unroll
    for (int j = 0; j < L::kJobs; ++j) {
      // the transition's value rows are the zeros written below
      if (SPLIT && ident && j >= kVJob0 && j < kVJob0 + L::kVJobs) continue;
      dma_job<L, TIn>(c, vrow, lds_l + b * L::kBytes, j, lane);
    }
  };
  // without a DMA wave: this compute wave's jobs wave + CW jj, jj in [j0, j1)
  constexpr int PER_WAVE = (L::kJobs + CW - 1) / CW;
  auto dma_share = [&](int ci, int b, int j0, int j1) __attribute__((always_inline)) {
    const ChunkSrc c = chunk_src<L>(u, ci, hk, hv, dv, ident ? 0 : col0, v, kin, qin, Kw, Tw, Sw, Pw);
#pragma unroll
    for (int jj = j0; jj < j1; ++jj) {
      const int j = wave + CW * jj;
      if (j >= L::kJobs || (SPLIT && ident && j >= kVJob0 && j < kVJob0 + L::kVJobs)) continue;
      dma_job<L, TIn>(c, vrow, lds_l + b * L::kBytes, j, lane);
    }
  };

  const int64_t sbase = (static_cast<int64_t>(u.n) * hv + u.h) * DK * ld + colw + lr;   // tile c: + 16 c
  if (SPLIT && ident) {
    // the transition's V tiles (both buffers) are zero
    for (int b = 0; b < L::kBuffers; ++b)
      for (int x = 16 * tid; x < L::kVBytes; x += 16 * static_cast<int>(blockDim.x))
        *reinterpret_cast<__attribute__((address_space(3))) u32x4*>(lds_l + b * L::kBytes + L::kOffV + x) =
            u32x4{0u, 0u, 0u, 0u};
  }
  const int nch = ce - cb;
  // The data waves and the compute waves run loops of their own with the same
  // barriers (two per chunk with one buffer, else one), so the state lives in
  // the compute waves' loop alone.
  if (data_wave) {
    if (dma_wave && nch > 0) {
      dma_chunk(cb, 0);
      wait_dma();
    }
    __syncthreads();
    for (int j = 0; j < nch; ++j) {
      const int b = L::kBuffers == 2 ? (j & 1) : 0;
      if (dma_wave && L::kBuffers == 2 && j + 1 < nch) {
        dma_chunk(cb + j + 1, b ^ 1);   // lands while the compute waves work on buffer b
        wait_dma();
      }
      if (L::kBuffers == 1) {
        __syncthreads();   // the compute waves are done with the only buffer
        if (dma_wave && j + 1 < nch) {
          dma_chunk(cb + j + 1, 0);
          wait_dma();
        }
      }
      __syncthreads();     // next chunk's operands are in LDS; this buffer is free
    }
    return;
  }

  f32x4 M[NC][NT];
  Frag mb[NC][DK / 32];
  f32x4 pout[4];
  if (SPLIT && ident) {
    // M0 = identity columns
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int td = 0; td < NT; ++td)
#pragma unroll
        for (int r = 0; r < 4; ++r) M[c][td][r] = (strow(td, lg, r) == colw + 16 * c + lr) ? 1.f : 0.f;
#pragma unroll
      for (int kk = 0; kk < DK / 32; ++kk) mb[c][kk] = chain_frag(M[c][2 * kk], M[c][2 * kk + 1]);
    }
  } else {
#pragma unroll
    for (int c = 0; c < NC; ++c)
      load_state<DK>(SPLIT ? nullptr : state_in, sbase + 16 * c, ld, lg, M[c], mb[c]);
  }
  if (!DMA_WAVE && nch > 0) {
    dma_share(cb, 0, 0, PER_WAVE);
    wait_dma();
  }
  __syncthreads();
  for (int j = 0; j < nch; ++j) {
    const int ci = cb + j;
    const int b = L::kBuffers == 2 ? (j & 1) : 0;
    if constexpr (FWD) {
      if (j > 0) store_chunk_out(o, u, ci - 1, hv, dv, colw, lane, pout);
    }
    const u32x4* pg = FWD ? Pw + (static_cast<int64_t>(u.slot0 + ci) * hv + u.h) * (2 * kTFrags * kWave) : nullptr;
    const unsigned char* buf = (const unsigned char*)(lds_l + b * L::kBytes);
    if constexpr (NC > 1) {
      // without a DMA wave: the next chunk's share, spread over the phases
      const bool prefetch = !DMA_WAVE && L::kBuffers == 2 && j + 1 < nch;
      constexpr int NPH = tiles_phases(DK);
      chunk_step_tiles<L, DK, NC>(buf, 16 * NC * wave, lane, M, mb, [&](int p) __attribute__((always_inline)) {
        const int j0 = p * PER_WAVE / NPH, j1 = (p + 1) * PER_WAVE / NPH;
        if (prefetch && j1 > j0) dma_share(ci + 1, b ^ 1, j0, j1);
      });
      if (!DMA_WAVE) wait_dma();   // this wave's share of the next chunk has landed
    } else {
      chunk_step<L, DK, FWD, false>(buf, 16 * wave, pg, lane, M[0], mb[0], pout, [](int) {});
    }
    if (L::kBuffers == 1) {
      __syncthreads();   // done with the only buffer
      if (!DMA_WAVE && j + 1 < nch) {
        dma_share(ci + 1, 0, 0, PER_WAVE);
        wait_dma();
      }
    }
    __syncthreads();     // next chunk's operands are in LDS (every wave's share)
  }
  if constexpr (FWD) {
    if (nch > 0) store_chunk_out(o, u, ce - 1, hv, dv, colw, lane, pout);
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    if (SPLIT && ident) {
      // the transition goes out transposed, A^T [d_k x d_k]: a lane's four
      // rows of its column are one 16-byte piece of that row of A^T
      float* at = dst + ((static_cast<int64_t>(u.n) * hv + u.h) * DK + colw + 16 * c + lr) * DK;
#pragma unroll
      for (int td = 0; td < NT; ++td) *reinterpret_cast<f32x4*>(at + strow(td, lg, 0)) = M[c][td];
    } else if (dst) {
#pragma unroll
      for (int td = 0; td < NT; ++td)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          dst[sbase + 16 * c + static_cast<int64_t>(strow(td, lg, r)) * ld] = M[c][td][r];
    }
  }
}

// LDS of the workgroup with outputs: chunk buffers (P read from global
// memory) and, per 16-column tile, the exchange from the recurrence wave to
// the output wave: Delta (4 KiB) and the split state (d_k / 32 x 2 KiB).
template <typename TIn, int DK, int TILES = 2>
struct ColsOutLayout {
  using L = ScanLds<TIn, DK, 16 * TILES, true, false>;
  static constexpr int kDBytes = 4 * kWave * 16;
  static constexpr int kMBytes = DK / 32 * 2 * kWave * 16;
  static constexpr int kTileBytes = kDBytes + kMBytes;
  static constexpr int kBuffers = 2 * L::kBytes + TILES * kTileBytes <= kLdsBytes ? 2 : 1;
  static constexpr int kOffX = kBuffers * L::kBytes;
  static constexpr int kBytes = kOffX + TILES * kTileBytes;
  static_assert(kBytes <= kLdsBytes, "column scan with outputs does not fit in LDS");
};

// One column-split workgroup with outputs (block `block` of `nblocks`), LDS in
// `lds_l`.  Two waves carry the recurrence of columns 16 c.. (chunk_step
// without outputs, exporting Delta before its region 5 and the split of M1 at
// its end) and two write the outputs of the same columns:
//   before the mid-chunk barrier: (Q M0)^T from the split M0 of the chunk;
//   after it: O^T = diag-scaled (Q M0)^T + Delta^T P^T, stored at the start
//   of the next chunk.
// With a DMA wave (bf16 inputs): wave 0 issues the next chunk's DMA (two
// thirds before the mid-chunk barrier, the rest after it), waves 1 + c carry
// the recurrence, waves 3 + c write the outputs; with waves assigned to SIMDs
// in turn, the DMA wave shares a SIMD with an output wave and each recurrence
// wave has one to itself.  Without (fp32 inputs): waves c carry the
// recurrence, waves 2 + c write the outputs and each issues half of the DMA.
// The products are those of chunk_step with outputs, in the same order, so the
// results are the same bit for bit.  TILES = 1 (bf16 inputs): a 16-column
// workgroup of a DMA wave, one recurrence wave and one output wave, for grids
// that fit on the chip at one workgroup per CU even so (each recurrence wave
// then has a CU's LDS bandwidth to itself).
template <typename TIn, int DK, int TILES = 2>
__device__ __forceinline__ void scan_cols_out_body(lds_byte* lds_l, int block, int nblocks,
                                                   const int32_t* __restrict__ cu, int32_t hk, int32_t hv,
                                                   int32_t dv, const TIn* __restrict__ v,
                                                   const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                                                   const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                                                   const float* __restrict__ Sw, const u32x4* __restrict__ Pw,
                                                   const float* __restrict__ state_in, TIn* __restrict__ o,
                                                   float* __restrict__ state_out,
                                                   const SeqOrder* order = nullptr) {
  using CL = ColsOutLayout<TIn, DK, TILES>;
  using L = typename CL::L;
  constexpr bool SPLIT = L::kSplit;
  constexpr int NT = DK / 16, NK = DK / 32;
  constexpr int NKA = ka_frags(DK);
  constexpr int NKF = L::kKFrags;
  constexpr bool DMA_WAVE = cols_dma_wave(true, SPLIT);
  static_assert(TILES == 2 || (TILES == 1 && DMA_WAVE), "one tile per workgroup needs the DMA wave");
  constexpr int kEarlyJobs = 2 * L::kJobs / 3;   // DMA jobs issued before the mid-chunk barrier
  static_assert(DMA_WAVE || (L::kKJobs % 2 == 0 && L::kTJobs % 2 == 0 && L::kPJobs == 0 &&
                             L::kVJobs % 2 == 0), "DMA halves need records of whole multiples of 2 KiB");
  constexpr int kHalf = (L::kKJobs + L::kTJobs + L::kVJobs) / 2;   // jobs per output wave, scalars aside
  const int tid = threadIdx.x;
  // wave index made provably uniform: DMA destinations (M0) stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int first_chain = DMA_WAVE ? 1 : 0;
  const bool dma_wave = DMA_WAVE && wave == 0;
  const bool chain_wave = wave >= first_chain && wave < first_chain + TILES;
  const bool out_wave = wave >= first_chain + TILES;
  const int tile = (wave - first_chain) % TILES, h = tile;
  const int lane = tid % kWave, lg = lane / 16, lr = lane % 16;
  constexpr int COLS = 16 * TILES;
  const int ngroups = dv / COLS;
  // logical unit: the column groups of a value head, then the value heads of a
  // key head, are adjacent and one cluster (same XCD, shared records in its L2)
  const int unit = xcd_cluster_remap(block, nblocks, ngroups * (hv / hk));
  const int col0 = COLS * (unit % ngroups);
  const ScanUnit u = scan_unit(cu, unit / (ngroups * hv), (unit / ngroups) % hv, hv, hk, order);
  const int colw = col0 + 16 * tile;
  const int64_t vrow = static_cast<int64_t>(hv) * dv;
  unsigned char* xd = (unsigned char*)(lds_l + CL::kOffX + tile * CL::kTileBytes);
  unsigned char* xm = xd + CL::kDBytes;

  // DMA jobs [j0, j1) of chunk ci into buffer b (the job index is a
  // compile-time constant in each instance, so every job is straight code)
  auto dma_jobs = [&](int ci, int b, auto j0c, auto j1c) __attribute__((always_inline)) {
    constexpr int j0 = decltype(j0c)::value, j1 = decltype(j1c)::value;
    const ChunkSrc c = chunk_src<L>(u, ci, hk, hv, dv, col0, v, kin, qin, Kw, Tw, Sw, Pw);
#pragma unroll
    for (int j = j0; j < j1; ++j) dma_job<L, TIn>(c, vrow, lds_l + b * L::kBytes, j, lane);
  };
  using J0 = std::integral_constant<int, 0>;
  using JE = std::integral_constant<int, kEarlyJobs>;
  using JN = std::integral_constant<int, L::kJobs>;
  // without a DMA wave: jobs 2 q + h of the K record, the T record and the V
  // rows for q in [q0, q1) (every record is a multiple of two jobs, so which
  // record a job reads is known at compile time); the scalars with the
  // second half
  auto dma_half = [&](int ci, int b, int q0, int q1) __attribute__((always_inline)) {
    const ChunkSrc c = chunk_src<L>(u, ci, hk, hv, dv, col0, v, kin, qin, Kw, Tw, Sw, Pw);
    lds_byte* dst = lds_l + b * L::kBytes;
#pragma unroll
    for (int q = q0; q < q1; ++q) {
      if (q < L::kKJobs / 2) {
        const int j = 2 * q + h;
        dma16_at(c.krec + 1024 * j, 16u * lane, dst + L::kOffK + 1024 * j);
      } else if (q < (L::kKJobs + L::kTJobs) / 2) {
        const int j = 2 * (q - L::kKJobs / 2) + h;
        dma16_at(c.trec + 1024 * j, 16u * lane, dst + L::kOffT + 1024 * j);
      } else {
        // V rows; pad rows repeat the last row (their beta is 0, so they add nothing)
        dma_rows<L::kVRowBytes>(static_cast<const TIn*>(c.v0), vrow, c.clen, dst + L::kOffV,
                                2 * (q - (L::kKJobs + L::kTJobs) / 2) + h, lane);
      }
    }
    if (q1 == kHalf) {
      if (h == 0) dma16_at(c.srow, 16u * lane, dst + L::kOffS);                       // bytes 0..1023
      else if (lane < 16) dma16_at(c.srow + 1024, 16u * lane, dst + L::kOffS + 1024); // 1024..1279
    }
  };

  f32x4 M[NT];
  Frag mb[NK];
  f32x4 pout[4];
  const int64_t sbase = (static_cast<int64_t>(u.n) * hv + u.h) * DK * dv + colw + lr;
  if (chain_wave) {
    load_state<DK>(state_in, sbase, dv, lg, M, mb);
    u32x4* x = reinterpret_cast<u32x4*>(xm);
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      x[(2 * kk) * kWave + lane] = __builtin_bit_cast(u32x4, mb[kk].hi);
      x[(2 * kk + 1) * kWave + lane] = __builtin_bit_cast(u32x4, mb[kk].lo);
    }
  } else if (u.nch > 0) {
    if (dma_wave) {
      dma_jobs(0, 0, J0{}, JN{});
      wait_dma();
    } else if (!DMA_WAVE) {
      dma_half(0, 0, 0, kHalf);
      wait_dma();
    }
  }
  __syncthreads();
  for (int ci = 0; ci < u.nch; ++ci) {
    const int b = CL::kBuffers == 2 ? (ci & 1) : 0;
    const unsigned char* base = (const unsigned char*)(lds_l + b * L::kBytes);
    const bool prefetch = CL::kBuffers == 2 && ci + 1 < u.nch;
    if (chain_wave) {
      chunk_step<L, DK, false, true>(base, 16 * tile, nullptr, lane, M, mb, pout,
                                     [](int k) __attribute__((always_inline)) {
                                       if (k == 5) lds_barrier();   // Delta is out
                                     },
                                     xd, xm);
    } else if (dma_wave) {
      if (prefetch) dma_jobs(ci + 1, b ^ 1, J0{}, JE{});
      lds_barrier();
      if (prefetch) dma_jobs(ci + 1, b ^ 1, JE{}, JN{});
    } else {
      if (ci > 0) store_chunk_out(o, u, ci - 1, hv, dv, colw, lane, pout);
      if (!DMA_WAVE && prefetch) dma_half(ci + 1, b ^ 1, 0, kHalf / 2);
      // (Q M0)^T: A = split M0 from the recurrence wave, B = Q fragments
      const u32x4* kf = reinterpret_cast<const u32x4*>(base + L::kOffK);
      const u32x4* x = reinterpret_cast<const u32x4*>(xm);
      Frag m0[NK];
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        m0[kk].hi = __builtin_bit_cast(bf16x8, x[(2 * kk) * kWave + lane]);
        m0[kk].lo = __builtin_bit_cast(bf16x8, x[(2 * kk + 1) * kWave + lane]);
      }
      // one token tile's Q fragments at a time (fp32 inputs carry hi and lo)
      f32x4 qm[4];
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        Frag qa[NK];
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
          const int f = NKA + ti * NK + kk;
          qa[kk].hi = __builtin_bit_cast(bf16x8, kf[f * kWave + kslot(lane)]);
          if constexpr (SPLIT) qa[kk].lo = __builtin_bit_cast(bf16x8, kf[(NKF + f) * kWave + kslot(lane)]);
        }
        qm[ti] = zero4();
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) qm[ti] = mma_b<SPLIT>(m0[kk], qa[kk], qm[ti]);
      }
      // P (split, six nonzero fragments) from global memory
      const u32x4* pg = Pw + (static_cast<int64_t>(u.slot0 + ci) * hv + u.h) * (2 * kTFrags * kWave);
      Frag pfr[kTFrags];
#pragma unroll
      for (int f = 0; f < kTFrags; ++f) {
        pfr[f].hi = __builtin_bit_cast(bf16x8, pg[f * kWave + lane]);
        pfr[f].lo = __builtin_bit_cast(bf16x8, pg[(kTFrags + f) * kWave + lane]);
      }
      lds_barrier();   // Delta is in
      const f32x4* xdv = reinterpret_cast<const f32x4*>(xd);
      f32x4 D[4];
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) D[ti] = xdv[ti * kWave + lane];
      const Frag dd0 = chain_frag(D[0], D[1]);
      const Frag dd1 = chain_frag(D[2], D[3]);
      const float* sc = reinterpret_cast<const float*>(base + L::kOffS);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        const float qe = sc[3 * kChunk + 16 * ti + lr];
#pragma unroll
        for (int r = 0; r < 4; ++r) pout[ti][r] = qe * qm[ti][r];
        pout[ti] = mma_x3(dd0, pfr[tri_frag(ti, 0)], pout[ti]);
        if (ti >= 2) pout[ti] = mma_x3(dd1, pfr[tri_frag(ti, 1)], pout[ti]);
      }
      if (!DMA_WAVE && prefetch) dma_half(ci + 1, b ^ 1, kHalf / 2, kHalf);
    }
    if (CL::kBuffers == 1) {
      __syncthreads();   // every wave is done with the only buffer
      if (ci + 1 < u.nch) {
        if (dma_wave) dma_jobs(ci + 1, 0, J0{}, JN{});
        else if (!DMA_WAVE && out_wave) dma_half(ci + 1, 0, 0, kHalf);
      }
    }
    if (dma_wave || (!DMA_WAVE && out_wave)) wait_dma();
    __syncthreads();     // next chunk's operands are in LDS; this buffer is free
  }
  if (out_wave) {
    if (u.nch > 0) store_chunk_out(o, u, u.nch - 1, hv, dv, colw, lane, pout);
  } else if (chain_wave && state_out) {
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        state_out[sbase + static_cast<int64_t>(strow(td, lg, r)) * dv] = M[td][r];
  }
}

template <typename TIn, int DK, bool FWD, int TILES = 2>
__global__ __launch_bounds__(cols_threads(FWD, sizeof(TIn) == 4, TILES)) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_scan_cols(const int32_t* __restrict__ cu, int32_t hk, int32_t hv, int32_t dv,
                 const TIn* __restrict__ v, const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                 const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                 const float* __restrict__ Sw, const u32x4* __restrict__ Pw,
                 const float* __restrict__ state_in, TIn* __restrict__ o, float* __restrict__ state_out) {
  if constexpr (FWD) {
    __shared__ __attribute__((aligned(1024))) unsigned char lds[ColsOutLayout<TIn, DK, TILES>::kBytes];
    scan_cols_out_body<TIn, DK, TILES>((lds_byte*)lds, blockIdx.x, gridDim.x, cu, hk, hv, dv, v, kin, qin, Kw, Tw,
                                       Sw, Pw, state_in, o, state_out);
  } else {
    using L = ColsLds<TIn, DK, false>;
    __shared__ __attribute__((aligned(1024))) unsigned char lds[L::kBuffers * L::kBytes];
    scan_cols_body<TIn, DK, false>((lds_byte*)lds, blockIdx.x, gridDim.x, cu, hk, hv, dv, v, kin, qin, Kw, Tw, Sw, Pw,
                                   state_in, o, state_out);
  }
}

// The 32-column scan with output waves over the P sequences `order` names
// (all of them, in index order, when its n is 0; grid P x Hv x d_v / 32, any
// number of rounds): the forward of the sequences peeled off a whole-head
// grid's partly empty last round, and of fp32 batches that do not fit on the
// chip (see launch_scan).
template <typename TIn, int DK>
__global__ __launch_bounds__(cols_threads(true, sizeof(TIn) == 4)) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_scan_cols_out_ord(const int32_t* __restrict__ cu, const SeqOrder order, int32_t hk, int32_t hv, int32_t dv,
                          const TIn* __restrict__ v, const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                          const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                          const float* __restrict__ Sw, const u32x4* __restrict__ Pw,
                          const float* __restrict__ state_in, TIn* __restrict__ o, float* __restrict__ state_out) {
  __shared__ __attribute__((aligned(1024))) unsigned char lds[ColsOutLayout<TIn, DK>::kBytes];
  scan_cols_out_body<TIn, DK>((lds_byte*)lds, blockIdx.x, gridDim.x, cu, hk, hv, dv, v, kin, qin, Kw, Tw, Sw, Pw,
                              state_in, o, state_out, &order);
}

// The wide column scan, tail replay only (grid N x Hv x d_v / COLS).
template <typename TIn, int DK, int COLS>
__global__ __launch_bounds__(cols_wide_threads(COLS)) __attribute__((amdgpu_waves_per_eu(COLS / 64, 2)))
void k_scan_cols_wide(const int32_t* __restrict__ cu, const SeqOrder order, int32_t hk, int32_t hv, int32_t dv,
                      const TIn* __restrict__ v, const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                      const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                      const float* __restrict__ Sw, float* __restrict__ state_out) {
  using L = ColsLds<TIn, DK, false, COLS>;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[L::kBuffers * L::kBytes];
  scan_cols_body<TIn, DK, false, COLS, kWhole, kWideTiles, false>((lds_byte*)lds, blockIdx.x, gridDim.x, cu, hk,
                                                                  hv, dv, v, kin, qin, Kw, Tw, Sw, nullptr,
                                                                  nullptr, nullptr, state_out, SplitOut{}, &order);
}

// Tail replay of bf16 inputs, 64 columns per workgroup: one 16-column tile per
// compute wave beside a DMA wave (the chains of the split scan's second half,
// which finish a chunk sooner than the wide scan's two-tile waves), grid
// P x Hv x d_v / 64 over the P sequences `order` names (all of them when its
// n is 0).  Used for batches whose grid takes at most three rounds of the
// chip, and for the sequences of a wide grid's partly empty last round.
template <typename TIn, int DK>
__global__ __launch_bounds__((kSplitCols2 / 16 + 1) * kWave)
void k_scan_cols_64(const int32_t* __restrict__ cu, const SeqOrder order, int32_t hk, int32_t hv, int32_t dv,
                      const TIn* __restrict__ v, const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                      const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                      const float* __restrict__ Sw, float* __restrict__ state_out) {
  using L = ColsLds<TIn, DK, false, kSplitCols2>;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[L::kBuffers * L::kBytes];
  scan_cols_body<TIn, DK, false, kSplitCols2, kWhole, 1, true>((lds_byte*)lds, blockIdx.x, gridDim.x, cu, hk, hv,
                                                               dv, v, kin, qin, Kw, Tw, Sw, nullptr, nullptr,
                                                               nullptr, state_out, SplitOut{}, &order);
}

// Tail replay in two halves, one launch: blocks [0, n_first) run the first
// half kSplitCols1 = 32 columns wide (grid N x Hv x d_v / 32; waves 3 and 4
// only take part in the barriers), the rest the second half and its
// transition kSplitCols2 = 64 columns wide (N x Hv x (d_v + d_k) / 64), one
// 16-column tile per compute wave.  state_out holds the first half's state
// until the combine runs.
constexpr int cols_split_threads() { return (kSplitCols2 / 16 + 1) * kWave; }
template <typename TIn, int DK>
__global__ __launch_bounds__(cols_split_threads())
void k_scan_cols_split(int32_t n_first, const int32_t* __restrict__ cu, int32_t hk, int32_t hv, int32_t dv,
                       const TIn* __restrict__ v, const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                       const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                       const float* __restrict__ Sw, float* __restrict__ state_out, float* __restrict__ m2,
                       float* __restrict__ a2) {
  using L1 = ColsLds<TIn, DK, false, kSplitCols1>;
  using L2 = ColsLds<TIn, DK, false, kSplitCols2>;
  constexpr int kB1 = L1::kBuffers * L1::kBytes, kB2 = L2::kBuffers * L2::kBytes;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[kB1 > kB2 ? kB1 : kB2];
  const int b = blockIdx.x;
  if (b < n_first)
    scan_cols_body<TIn, DK, false, kSplitCols1, kFirstHalf>((lds_byte*)lds, b, n_first, cu, hk, hv, dv, v, kin, qin,
                                                            Kw, Tw, Sw, nullptr, nullptr, nullptr, state_out);
  else
    scan_cols_body<TIn, DK, false, kSplitCols2, kSecondHalf>((lds_byte*)lds, b - n_first,
                                                             static_cast<int>(gridDim.x) - n_first, cu, hk, hv, dv, v,
                                                             kin, qin, Kw, Tw, Sw, nullptr, nullptr, nullptr, nullptr,
                                                             SplitOut{m2, a2});
}

// state = A state + B per (sequence, value head): A^T [d_k x d_k], state and
// B [d_k x d_v], fp32 row-major.  grid N x Hv x d_v / 16; a workgroup owns 16
// whole columns of one state (it reads them all before it writes any) and
// stages those columns in LDS, every load in flight at once.  The product
// runs on fp32 MFMA (16x16x4, fp32 products and sums): wave w takes the
// 16-row tiles w, w + 4, ..; per 4-step slice of k, lane l supplies
// A[16 t + l % 16][k + l / 16] (= A^T[k + l / 16][..], read from memory into
// registers up front) and column l % 16 of row k + l / 16 of the staged
// state, and holds D[4 (l / 16) + i][l % 16] of the tile.  With 8 KiB of LDS
// the combine leaves room for four preparation workgroups per CU beside it
// in k_combine_intra.
constexpr int kCombineThreads = 256;
constexpr int kCombineCols = 16;
template <int DK>
struct CombineLds {
  alignas(16) float ms[DK * kCombineCols];
};

// `block` of `nblocks`: the column groups of one (sequence, head) are one
// cluster on one XCD, so the head's transition is fetched from memory once
// and its other workgroups find it in that XCD's L2.
template <int DK>
__device__ __forceinline__ void combine_body(CombineLds<DK>& sm, int block, int nblocks, int32_t dv,
                                             const float* __restrict__ At, const float* __restrict__ B,
                                             float* __restrict__ state) {
  constexpr int PER = DK * kCombineCols / kCombineThreads;   // staged column values per thread
  constexpr int TILES = DK / 16 / (kCombineThreads / kWave);  // row tiles per wave
  float* ms = sm.ms;
  const int groups = dv / kCombineCols;
  const int unit = xcd_cluster_remap(block, nblocks, groups);
  const int64_t head = unit / groups;
  const int c0 = kCombineCols * (unit % groups);
  const int tid = threadIdx.x, wave = tid / kWave, lane = tid % kWave;
  const int li = lane % 16, lk = lane / 16;
  float* st = state + head * DK * dv + c0;
  const float* bm = B + head * DK * dv + c0;
  const float* at = At + head * DK * DK;
  // the wave's A operands straight from memory (A^T rows are 16 consecutive
  // floats per tile: 64-byte pieces), every load in flight at once
  float av[DK / 4][TILES];
#pragma unroll
  for (int k = 0; k < DK; k += 4)
#pragma unroll
    for (int t = 0; t < TILES; ++t) av[k / 4][t] = at[(k + lk) * DK + 16 * (wave + 4 * t) + li];
  float mv[PER];
#pragma unroll
  for (int i = 0; i < PER; ++i) {
    const int x = tid + kCombineThreads * i;
    mv[i] = st[static_cast<int64_t>(x / kCombineCols) * dv + x % kCombineCols];
  }
  f32x4 acc[TILES];
#pragma unroll
  for (int t = 0; t < TILES; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i)
      acc[t][i] = bm[static_cast<int64_t>(16 * (wave + 4 * t) + 4 * lk + i) * dv + li];
#pragma unroll
  for (int i = 0; i < PER; ++i) ms[tid + kCombineThreads * i] = mv[i];
  __syncthreads();
#pragma unroll
  for (int k = 0; k < DK; k += 4) {
    const float b = ms[(k + lk) * kCombineCols + li];
#pragma unroll
    for (int t = 0; t < TILES; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[k / 4][t], b, acc[t], 0, 0, 0);
  }
#pragma unroll
  for (int t = 0; t < TILES; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) st[static_cast<int64_t>(16 * (wave + 4 * t) + 4 * lk + i) * dv + li] = acc[t][i];
}
template <int DK>
__global__ __launch_bounds__(kCombineThreads)
void k_state_combine(int32_t dv, const float* __restrict__ At, const float* __restrict__ B,
                     float* __restrict__ state) {
  __shared__ CombineLds<DK> sm;
  combine_body<DK>(sm, blockIdx.x, gridDim.x, dv, At, B, state);
}

// The combine of a split tail replay beside the suffix's chunk preparation,
// one launch: blocks [0, n_comb) run k_state_combine, the rest k_intra for the
// suffix chunks (with outputs).  The combine is short and light, so the
// preparation workgroups fill the chip around it.  No workgroup waits for
// another.
template <typename TIn, int DK>
__global__ __launch_bounds__(kCombineThreads)
void k_combine_intra(int32_t n_comb, int32_t dv, const float* __restrict__ At, const float* __restrict__ B,
                     float* __restrict__ state, int32_t slots_s, const int32_t* __restrict__ cu_s, int32_t num_seqs,
                     int32_t hk, int32_t hv, const TIn* __restrict__ q_s, const TIn* __restrict__ k_s,
                     const float* __restrict__ g_s, const float* __restrict__ beta_s, float scale,
                     u32x4* __restrict__ Kw_s, u32x4* __restrict__ Tw_s, float* __restrict__ Sw_s,
                     u32x4* __restrict__ Pw_s) {
  static_assert(kCombineThreads == 4 * kWave, "the preparation body runs on four waves");
  using LC = CombineLds<DK>;
  using LI = IntraLds<TIn, DK, true>;
  constexpr size_t kBytes = sizeof(LC) > sizeof(LI) ? sizeof(LC) : sizeof(LI);
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kBytes];
  const int b = blockIdx.x;
  if (b < n_comb) {
    combine_body<DK>(*reinterpret_cast<LC*>(smem), b, n_comb, dv, At, B, state);
  } else {
    const int i = b - n_comb;
    int slot, h;
    intra_unit(i, slots_s * hv, hv, hv / hk, slot, h);
    intra_body<TIn, DK, true>(*reinterpret_cast<LI*>(smem), slot, h, cu_s, num_seqs, hk, hv,
                              q_s, k_s, g_s, beta_s, scale, Kw_s, Tw_s, Sw_s, Pw_s);
  }
}

// ---------------------------------------------------------------- replay scan + suffix intra
// One launch, two kinds of workgroup (256 threads): blocks [0, n_scan) run the
// column-split tail replay (FWD = false, zero start, final state to
// `state_mid`; the fourth wave only takes part in the barriers), the rest run
// k_intra for the suffix chunks (with outputs), so the suffix's records are
// built on the CUs the replay leaves idle.  No workgroup waits for another.
template <typename TIn, int DK>
__global__ __launch_bounds__(4 * kWave) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_scan_cols_intra(int32_t n_scan, const int32_t* __restrict__ cu_t, int32_t hk, int32_t hv, int32_t dv,
                       const TIn* __restrict__ v_t, const TIn* __restrict__ k_t, const u32x4* __restrict__ Kw_t,
                       const u32x4* __restrict__ Tw_t, const float* __restrict__ Sw_t,
                       float* __restrict__ state_mid,
                       int32_t slots_s, const int32_t* __restrict__ cu_s, int32_t num_seqs,
                       const TIn* __restrict__ q_s, const TIn* __restrict__ k_s,
                       const float* __restrict__ g_s, const float* __restrict__ beta_s, float scale,
                       u32x4* __restrict__ Kw_s, u32x4* __restrict__ Tw_s, float* __restrict__ Sw_s,
                       u32x4* __restrict__ Pw_s) {
  using LS = ColsLds<TIn, DK, false>;
  using LI = IntraLds<TIn, DK, true>;
  constexpr size_t kScanBytes = static_cast<size_t>(LS::kBuffers) * LS::kBytes;
  constexpr size_t kBytes = kScanBytes > sizeof(LI) ? kScanBytes : sizeof(LI);
  __shared__ __attribute__((aligned(1024))) unsigned char smem[kBytes];
  if (static_cast<int>(blockIdx.x) < n_scan) {
    scan_cols_body<TIn, DK, false>((lds_byte*)smem, blockIdx.x, n_scan, cu_t, hk, hv, dv, v_t, k_t, nullptr, Kw_t,
                                   Tw_t,
                                   Sw_t, nullptr, nullptr, nullptr, state_mid);
  } else {
    const int i = blockIdx.x - n_scan;
    int slot, h;
    intra_unit(i, slots_s * hv, hv, hv / hk, slot, h);
    intra_body<TIn, DK, true>(*reinterpret_cast<LI*>(smem), slot, h, cu_s, num_seqs, hk, hv,
                              q_s, k_s, g_s, beta_s, scale, Kw_s, Tw_s, Sw_s, Pw_s);
  }
}

// ---------------------------------------------------------------- throughput kernel
// grid = N x Hv: d_v/16 waves (two per SIMD for d_v = 128), each 16 columns,
// sharing one copy of the chunk's records per head; every wave issues an equal
// share of the next chunk's DMA, spread over the chunk's regions.  Used when
// the latency kernel's grid would not fit on the chip at once.
constexpr int head_threads(int dv) { return dv / 16 * kWave; }

template <typename TIn, int DK, int DV, bool FWD>
__global__ __launch_bounds__(head_threads(DV))
void k_scan_head(const int32_t* __restrict__ cu, const SeqOrder order, int32_t hk, int32_t hv,
                 const TIn* __restrict__ v, const TIn* __restrict__ kin, const TIn* __restrict__ qin,
                 const u32x4* __restrict__ Kw, const u32x4* __restrict__ Tw,
                 const float* __restrict__ Sw, const u32x4* __restrict__ Pw,
                 const float* __restrict__ state_in, TIn* __restrict__ o, float* __restrict__ state_out) {
  using L = ScanLds<TIn, DK, DV, FWD, false>;
  constexpr int NT = DK / 16;
  constexpr int W = DV / 16;
  constexpr int PER_WAVE = (L::kJobs + W - 1) / W;   // DMA jobs per wave per chunk
  __shared__ __attribute__((aligned(1024))) unsigned char lds_g[L::kBuffers * L::kBytes];
  lds_byte* lds = (lds_byte*)lds_g;
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave, lg = lane / 16, lr = lane % 16;
  // logical unit: the value heads of a key head are adjacent and one cluster (same XCD)
  const int unit = xcd_cluster_remap(blockIdx.x, gridDim.x, hv / hk);
  const ScanUnit u = scan_unit(cu, unit / hv, unit % hv, hv, hk, &order);
  const int col = 16 * wave + lr;
  const int64_t vrow = static_cast<int64_t>(hv) * DV;
  // jobs wave + W * jj, jj in [j0, j1), of chunk ci into buffer b
  auto dma_share = [&](int ci, int b, int j0, int j1) __attribute__((always_inline)) {
    const ChunkSrc c = chunk_src<L>(u, ci, hk, hv, DV, 0, v, kin, qin, Kw, Tw, Sw, Pw);
#pragma unroll
    for (int jj = j0; jj < j1; ++jj) {
      const int j = wave + W * jj;
      if (j < L::kJobs) dma_job<L, TIn>(c, vrow, lds + b * L::kBytes, j, lane);
    }
  };

  f32x4 M[NT];
  Frag mb[DK / 32];
  f32x4 pout[4];
  const int64_t sbase = (static_cast<int64_t>(u.n) * hv + u.h) * DK * DV + col;
  load_state<DK>(state_in, sbase, DV, lg, M, mb);

  if (u.nch > 0) {
    dma_share(0, 0, 0, PER_WAVE);
    wait_dma();
  }
  __syncthreads();
  for (int ci = 0; ci < u.nch; ++ci) {
    const int b = L::kBuffers == 2 ? (ci & 1) : 0;
    if constexpr (FWD) {
      if (ci > 0) store_chunk_out(o, u, ci - 1, hv, DV, col - lr, lane, pout);
    }
    const bool prefetch = L::kBuffers == 2 && ci + 1 < u.nch;
    // the next chunk's DMA share, a few jobs at the start of each region
    auto hook = [&](int k) __attribute__((always_inline)) {
      if (prefetch) {
        const int j0 = k * PER_WAVE / 7, j1 = (k + 1) * PER_WAVE / 7;
        if (j1 > j0) dma_share(ci + 1, b ^ 1, j0, j1);
      }
    };
    const u32x4* pg = FWD ? Pw + (static_cast<int64_t>(u.slot0 + ci) * hv + u.h) * (2 * kTFrags * kWave) : nullptr;
    chunk_step<L, DK, FWD, false>((const unsigned char*)(lds + b * L::kBytes), 16 * wave, pg, lane, M, mb, pout,
                                  hook);
    if (L::kBuffers == 1) {
      __syncthreads();   // every wave is done with the only buffer
      if (ci + 1 < u.nch) dma_share(ci + 1, 0, 0, PER_WAVE);
    }
    wait_dma();          // this wave's share of the next chunk has landed
    __syncthreads();     // ... and everyone else's; this chunk's buffer is free
  }
  if constexpr (FWD) {
    if (u.nch > 0) store_chunk_out(o, u, u.nch - 1, hv, DV, col - lr, lane, pout);
  }
  if (state_out) {
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        state_out[sbase + static_cast<int64_t>(strow(td, lg, r)) * DV] = M[td][r];
  }
}

}  // namespace gdn
