// Chunk scan kernel: the sequential part of the recurrence.
//
// One workgroup per (sequence, value head, 32 state columns): two compute waves
// each own 16 columns of M = S^T (d_k x d_v) and keep them in registers for the
// whole sequence, and a third wave only moves data.  Per 64-token chunk, with
// M0 the state at chunk start:
//   R      = diag(beta) V - diag(beta e^G) (K M0)
//   Delta  = T R                                                  (T from k_intra)
//   O      = diag(scale e^G) (Q M0) + P Delta                     (outputs only)
//   M1     = e^{G_last} M0 + K^T diag(e^{G_last - G}) Delta
// All four products run on MFMA.  The contraction order inside every 32-wide k
// step is permuted (kperm) so each accumulator is directly the next product's
// B operand.  fp32 operands (M0, R, Delta, T, P) are split into bf16 hi + lo.
//
// Every A operand (K, K^T, Q, T, P) comes from a workspace record that k_intra
// wrote in fragment order, so a compute wave fetches each operand with one
// conflict-free 16-byte LDS read per lane.  The data wave copies the next
// chunk's records and value rows global -> LDS by DMA (global_load_lds, 16
// bytes per lane) into one of two LDS buffers while the compute waves work on
// the other; the compute waves issue each group of LDS reads one MFMA group
// ahead of its use, so LDS latency hides behind the matrix cores.
#pragma once

#include "gdn_device.h"
#include "gdn_intra.h"
#include "gdn_plan.h"

namespace gdn {

constexpr int kLdsBytes = 160 * 1024;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// 16 bytes per lane from `src` (per lane) to LDS `dst + 16 * lane` (dst uniform).
__device__ __forceinline__ void dma16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)dst, 16, 0, 0);
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Byte offset of byte `byte_in_row` of row `row` in a row tile whose rows hold
// ROW_BYTES / 16 pieces of 16 bytes, piece p of row R stored at p ^ (R % pieces).
template <int ROW_BYTES>
__device__ __forceinline__ int swz(int row, int byte_in_row) {
  constexpr int pieces = ROW_BYTES / 16;
  return row * ROW_BYTES + 16 * ((byte_in_row / 16) ^ (row % pieces)) + byte_in_row % 16;
}

constexpr int kComputeWaves = 2;
constexpr int kScanCols = 16 * kComputeWaves;              // state columns per workgroup
constexpr int kScanThreads = (kComputeWaves + 1) * kWave;   // + the data wave

// LDS layout of one chunk buffer.
template <typename TIn, int DK, bool FWD>
struct ScanLds {
  static constexpr bool kSplit = sizeof(TIn) == 4;
  static constexpr int kKFrags = k_record_frags(DK, FWD);         // per bf16 part
  static constexpr int kKBytes = static_cast<int>(k_record_bytes(DK, FWD, kSplit));
  static constexpr int kTBytes = static_cast<int>(kTRecordBytes);
  static constexpr int kPBytes = FWD ? static_cast<int>(kPRecordBytes) : 0;
  static constexpr int kSBytes = static_cast<int>(kSRecordBytes);
  static constexpr int kVRowBytes = kScanCols * static_cast<int>(sizeof(TIn));
  static constexpr int kVBytes = kChunk * kVRowBytes;
  static constexpr int kOffK = 0;                 // K record
  static constexpr int kOffT = kOffK + kKBytes;
  static constexpr int kOffP = kOffT + kTBytes;
  static constexpr int kOffS = kOffP + kPBytes;
  static constexpr int kOffV = kOffS + kSBytes;
  static constexpr int kBytes = kOffV + kVBytes;
  static constexpr int kBuffers = 2 * kBytes <= kLdsBytes ? 2 : 1;
  static constexpr int kVBlocks = kVBytes / 1024;
};

// DMA of rows [0, 64) of a token-major tensor (row 0 at `row0`, 1 KiB block
// `blk` of the tile) into a swizzled LDS row tile; rows past `rows` repeat the
// last valid row.
template <int ROW_BYTES, typename T>
__device__ __forceinline__ void dma_rows(const T* row0, int64_t row_stride, int rows, unsigned char* dst,
                                         int blk, int lane) {
  constexpr int pieces = ROW_BYTES / 16;
  constexpr int rows_per_block = 1024 / ROW_BYTES;
  const int r = blk * rows_per_block + lane / pieces;
  const int p = (lane % pieces) ^ (r % pieces);
  const T* src = row0 + min(r, rows - 1) * row_stride + p * (16 / static_cast<int>(sizeof(T)));
  dma16(src, dst + blk * 1024);
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
__device__ __forceinline__ void store_out(__amdgpu_buffer_rsrc_t r, int voff, int soff, float x, uint16_t*) {
  const uint32_t w = __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{x, 0.f}, bf16x2));
  __builtin_amdgcn_raw_buffer_store_b16(static_cast<uint16_t>(w), r, voff, soff, 0);
}
__device__ __forceinline__ void store_out(__amdgpu_buffer_rsrc_t r, int voff, int soff, float x, float*) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, x), r, voff, soff, 0);
}

template <typename TIn, int DK, bool FWD>
__global__ __launch_bounds__(kScanThreads) __attribute__((amdgpu_waves_per_eu(1, 1)))
void k_scan(const int32_t* __restrict__ cu, int32_t hk, int32_t hv, int32_t dv,
            const TIn* __restrict__ v,
            const u32x4* __restrict__ Kw,
            const u32x4* __restrict__ Tw,
            const float* __restrict__ Sw,
            const u32x4* __restrict__ Pw,
            const float* __restrict__ state_in,
            TIn* __restrict__ o,
            float* __restrict__ state_out) {
  using L = ScanLds<TIn, DK, FWD>;
  constexpr bool SPLIT = L::kSplit;
  constexpr int NT = DK / 16;         // 16-row tiles of M
  constexpr int NK = DK / 32;         // 32-wide k steps over d_k
  constexpr int NKA = ka_frags(DK), NKT = kt_frags(DK);
  constexpr int NKF = L::kKFrags;
  constexpr int VRB = L::kVRowBytes;
  __shared__ __attribute__((aligned(1024))) unsigned char lds[L::kBuffers * L::kBytes];

  const int tid = threadIdx.x;
  // wave index made provably uniform: DMA destinations (M0) stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const bool data_wave = wave == kComputeWaves;
  const int lane = tid % kWave;
  const int lg = lane / 16, lr = lane % 16;
  const int ngroups = dv / kScanCols;
  // logical unit: the column groups of a value head, then the value heads of a
  // key head, are adjacent (same XCD, shared records in its L2)
  const int unit = xcd_remap(blockIdx.x, gridDim.x);
  const int cgrp = unit % ngroups;
  const int h = (unit / ngroups) % hv;
  const int n = unit / (ngroups * hv);
  const int kh = h / (hv / hk);
  const int col0 = kScanCols * cgrp;           // first state column of the workgroup
  const int wcol = 16 * wave + lr;             // this lane's column within the workgroup
  const int col = col0 + wcol;
  const int tok0 = cu[n];
  const int len = cu[n + 1] - tok0;
  const int slot0 = tok0 / kChunk + n;
  const int nch = (len + kChunk - 1) / kChunk;
  const int64_t vrow = static_cast<int64_t>(hv) * dv;   // token stride of v and o

  // ---- the data wave copies chunk ci's operands into LDS buffer b
  auto dma_chunk = [&](int ci, int b) __attribute__((always_inline)) {
    unsigned char* base = lds + b * L::kBytes;
    const int64_t srec = static_cast<int64_t>(slot0 + ci);
    const int t0 = tok0 + ci * kChunk;
    const int clen = min(kChunk, len - ci * kChunk);
    const unsigned char* krec = reinterpret_cast<const unsigned char*>(Kw) + (srec * hk + kh) * L::kKBytes;
    const unsigned char* trec = reinterpret_cast<const unsigned char*>(Tw) + (srec * hv + h) * L::kTBytes;
    const unsigned char* prec = reinterpret_cast<const unsigned char*>(Pw) + (srec * hv + h) * L::kPBytes;
    // records: 1 KiB blocks copied verbatim, fully unrolled (one DMA each)
#pragma unroll
    for (int blk = 0; blk < L::kKBytes / 1024; ++blk) dma16(krec + 1024 * blk + 16 * lane, base + L::kOffK + 1024 * blk);
#pragma unroll
    for (int blk = 0; blk < L::kTBytes / 1024; ++blk) dma16(trec + 1024 * blk + 16 * lane, base + L::kOffT + 1024 * blk);
#pragma unroll
    for (int blk = 0; blk < L::kPBytes / 1024; ++blk) dma16(prec + 1024 * blk + 16 * lane, base + L::kOffP + 1024 * blk);
    // row scalars: 1280 bytes = one full block and a quarter block
    const unsigned char* srow = reinterpret_cast<const unsigned char*>(Sw) + (srec * hv + h) * L::kSBytes;
    dma16(srow + 16 * lane, base + L::kOffS);
    if (lane < 16) dma16(srow + 1024 + 16 * lane, base + L::kOffS + 1024);
    // V rows, this workgroup's columns (pad rows repeat the last row; their beta
    // is 0, so they add nothing)
    const TIn* v0 = v + static_cast<int64_t>(t0) * vrow + static_cast<int64_t>(h) * dv + col0;
#pragma unroll
    for (int blk = 0; blk < L::kVBlocks; ++blk) dma_rows<VRB>(v0, vrow, clen, base + L::kOffV, blk, lane);
  };

  // state M (compute waves), accumulator layout: M[td][r] = M[16 td + 4 lg + r][col]
  f32x4 M[NT];
  const int64_t sbase = (static_cast<int64_t>(n) * hv + h) * DK * dv + col;
  if (!data_wave && state_in != nullptr) {
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 4; ++r) M[td][r] = state_in[sbase + static_cast<int64_t>(16 * td + 4 * lg + r) * dv];
  } else {
#pragma unroll
    for (int td = 0; td < NT; ++td) M[td] = zero4();
  }
  // M split into bf16 hi/lo as the B operand of K M0 (and Q M0), one per k step;
  // refreshed at the end of every chunk's state update
  Frag mb[NK];
#pragma unroll
  for (int kk = 0; kk < NK; ++kk) mb[kk] = chain_frag(M[2 * kk], M[2 * kk + 1]);

  if (data_wave && nch > 0) {
    dma_chunk(0, 0);
    wait_dma();
  }
  __syncthreads();

  for (int ci = 0; ci < nch; ++ci) {
    const int b = L::kBuffers == 2 ? (ci & 1) : 0;
    if (data_wave) {
      if (L::kBuffers == 2 && ci + 1 < nch) {
        dma_chunk(ci + 1, b ^ 1);   // lands while the compute waves work on buffer b
        wait_dma();
      }
    } else {
      const unsigned char* base = lds + b * L::kBytes;
      const u32x4* kf = reinterpret_cast<const u32x4*>(base + L::kOffK);
      const u32x4* tf = reinterpret_cast<const u32x4*>(base + L::kOffT);
      const u32x4* pf = reinterpret_cast<const u32x4*>(base + L::kOffP);
      const float* sc = reinterpret_cast<const float*>(base + L::kOffS);
      const unsigned char* vtile = base + L::kOffV;
      const int t0 = tok0 + ci * kChunk;
      const int clen = min(kChunk, len - ci * kChunk);
      // fragment f of the K record (`nf` fragments per bf16 part; the lo part
      // exists for fp32 inputs only)
      auto ldf = [&](Frag& x, const u32x4* rec, int f, int nf) __attribute__((always_inline)) {
        x.hi = __builtin_bit_cast(bf16x8, rec[f * kWave + lane]);
        if constexpr (SPLIT) x.lo = __builtin_bit_cast(bf16x8, rec[(nf + f) * kWave + lane]);
      };
      // fp32-derived records (T, P): always hi and lo
      auto ld_split = [&](Frag& x, const u32x4* rec, int f) __attribute__((always_inline)) {
        x.hi = __builtin_bit_cast(bf16x8, rec[f * kWave + lane]);
        x.lo = __builtin_bit_cast(bf16x8, rec[(kTFrags + f) * kWave + lane]);
      };
      // K (and Q) operands of row tiles 2 tp, 2 tp + 1 for every k step
      auto ld_ka = [&](Frag (&a)[2][NK], Frag (&aq)[2][NK], int tp) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int kk = 0; kk < NK; ++kk) {
            ldf(a[u][kk], kf, (2 * tp + u) * NK + kk, NKF);
            if constexpr (FWD) ldf(aq[u][kk], kf, NKA + NKT + (2 * tp + u) * NK + kk, NKF);
          }
      };
      // K^T operands of every row tile of M for k step kk
      auto ld_kt = [&](Frag (&a)[NT], int kk) __attribute__((always_inline)) {
#pragma unroll
        for (int td = 0; td < NT; ++td) ldf(a[td], kf, NKA + 2 * td + kk, NKF);
      };

      // The chunk runs as a chain of regions.  Each region issues the LDS reads of
      // a later region, runs MFMAs on operands that are ready, and does VALU work
      // (scaling, hi/lo splits) for the next region, independent of its own MFMAs
      // so the two overlap.
      Frag ka0[2][NK], qa0[2][NK], ka1[2][NK], qa1[2][NK];
      Frag tfr[kTFrags], pfr[FWD ? kTFrags : 1];
      Frag kt0[NT], kt1[NT];
      f32x4 km[4], qm[4], acc[NT], bv[4], R[4], D[4];
      u32x2 vraw[4];
      float vf[4][4];

      // ---- region 0: first operands
      ld_ka(ka0, qa0, 0);
      if constexpr (!SPLIT) {
        // transposing read: lane (g, c) gets V[16 ti + 4 g + r][c], r = 0..3
#pragma unroll
        for (int ti = 0; ti < 4; ++ti)
          vraw[ti] = lds_read_tr16(vtile + swz<VRB>(16 * ti + 4 * lg + lr / 4, 2 * (16 * wave + 4 * (lr % 4))));
      } else {
#pragma unroll
        for (int ti = 0; ti < 4; ++ti)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            vf[ti][r] = *reinterpret_cast<const float*>(vtile + swz<VRB>(16 * ti + 4 * lg + r, 4 * wcol));
      }
      ld_ka(ka1, qa1, 1);
      __builtin_amdgcn_sched_barrier(0);

      // ---- region 1: K M0 for row tiles 0, 1 | beta V, e^{G_last} M0
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        km[u] = zero4();
        qm[u] = zero4();
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
          km[u] = mma_a<SPLIT>(ka0[u][kk], mb[kk], km[u]);
          if constexpr (FWD) qm[u] = mma_a<SPLIT>(qa0[u][kk], mb[kk], qm[u]);
        }
      }
      {
        const float eg = sc[4 * kChunk];
#pragma unroll
        for (int ti = 0; ti < 4; ++ti) {
          const f32x4 bta = *reinterpret_cast<const f32x4*>(sc + 0 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
          for (int r = 0; r < 4; ++r) bv[ti][r] = bta[r] * (SPLIT ? vf[ti][r] : bf16_elt(vraw[ti], r));
        }
#pragma unroll
        for (int td = 0; td < NT; ++td)
#pragma unroll
          for (int r = 0; r < 4; ++r) acc[td][r] = eg * M[td][r];
      }
      __builtin_amdgcn_sched_barrier(0);

      // ---- region 2: K M0 for row tiles 2, 3 | R rows 0..31 and their split;
      //      T arrives
#pragma unroll
      for (int f = 0; f < kTFrags; ++f) ld_split(tfr[f], tf, f);
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        km[2 + u] = zero4();
        qm[2 + u] = zero4();
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
          km[2 + u] = mma_a<SPLIT>(ka1[u][kk], mb[kk], km[2 + u]);
          if constexpr (FWD) qm[2 + u] = mma_a<SPLIT>(qa1[u][kk], mb[kk], qm[2 + u]);
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

      // ---- region 3: Delta = T R, k step 0 for all row tiles | R rows 32..63
      //      and their split; K^T (k step 0) arrives
      ld_kt(kt0, 0);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) D[ti] = mma_x3(tfr[tri_frag(ti, 0)], rb0, zero4());
      make_r(2);
      make_r(3);
      const Frag rb1 = chain_frag(R[2], R[3]);
      __builtin_amdgcn_sched_barrier(0);

      // ---- region 4: Delta, k step 1 for row tiles 2, 3 | split of the
      //      weighted Delta rows 0..31 (and of Delta for the outputs); K^T
      //      arrives
      ld_kt(kt1, 1);
#pragma unroll
      for (int ti = 2; ti < 4; ++ti) D[ti] = mma_x3(tfr[tri_frag(ti, 1)], rb1, D[ti]);
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

      // ---- region 5: M1 partial, k step 0 (tokens 0..31) | split of the
      //      weighted Delta rows 32..63; P (outputs) arrives
      if constexpr (FWD) {
#pragma unroll
        for (int f = 0; f < kTFrags; ++f) ld_split(pfr[f], pf, f);
      }
#pragma unroll
      for (int td = 0; td < NT; ++td) acc[td] = mma_a<SPLIT>(kt0[td], db0, acc[td]);
      make_dw(2);
      make_dw(3);
      const Frag db1 = chain_frag(Dw[2], Dw[3]);
      Frag dd1;
      if constexpr (FWD) dd1 = chain_frag(D[2], D[3]);
      __builtin_amdgcn_sched_barrier(0);

      // ---- outputs O = scale e^G (Q M0) + P Delta; rows past the chunk's end
      //      fall outside the buffer range and are not written
      if constexpr (FWD) {
        constexpr int E = static_cast<int>(sizeof(TIn));
        const int row_bytes = static_cast<int>(vrow) * E;
        const __amdgpu_buffer_rsrc_t orsrc =
            out_rsrc(o + static_cast<int64_t>(t0) * vrow + static_cast<int64_t>(h) * dv, clen * row_bytes);
        const int voff = 4 * lg * row_bytes + col * E;
        f32x4 out[4];
#pragma unroll
        for (int ti = 0; ti < 4; ++ti) {
          const f32x4 qe = *reinterpret_cast<const f32x4*>(sc + 3 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
          for (int r = 0; r < 4; ++r) out[ti][r] = qe[r] * qm[ti][r];
          out[ti] = mma_x3(pfr[tri_frag(ti, 0)], dd0, out[ti]);
          if (ti >= 2) out[ti] = mma_x3(pfr[tri_frag(ti, 1)], dd1, out[ti]);
        }
#pragma unroll
        for (int ti = 0; ti < 4; ++ti)
#pragma unroll
          for (int r = 0; r < 4; ++r) store_out(orsrc, voff + (16 * ti + r) * row_bytes, 0, out[ti][r], o);
        __builtin_amdgcn_sched_barrier(0);
      }

      // ---- region 6: M1, k step 1 (tokens 32..63) | split of M1 for the next chunk
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        M[2 * kk] = mma_a<SPLIT>(kt1[2 * kk], db1, acc[2 * kk]);
        M[2 * kk + 1] = mma_a<SPLIT>(kt1[2 * kk + 1], db1, acc[2 * kk + 1]);
        mb[kk] = chain_frag(M[2 * kk], M[2 * kk + 1]);
      }
    }

    if (L::kBuffers == 1) {
      __syncthreads();   // the compute waves are done with the only buffer
      if (data_wave && ci + 1 < nch) {
        dma_chunk(ci + 1, 0);
        wait_dma();
      }
    }
    __syncthreads();     // next chunk's operands are in LDS; this buffer is free
  }

  if (!data_wave && state_out) {
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        state_out[sbase + static_cast<int64_t>(16 * td + 4 * lg + r) * dv] = M[td][r];
  }
}

}  // namespace gdn
