// Chunk scan kernel: the sequential part of the recurrence.
//
// One workgroup per (sequence, value head, 32 state columns); each of its two
// waves owns 16 columns of M = S^T (d_k x d_v) and keeps them in registers for
// the whole sequence.  Per 64-token chunk, with M0 the state at chunk start:
//   R      = diag(beta) V - diag(beta e^G) (K M0)                 (64 x 16)
//   Delta  = T R                                                  (T from k_intra)
//   O      = diag(scale e^G) (Q M0) + P Delta                     (outputs only)
//   M1     = e^{G_last} M0 + K^T diag(e^{G_last - G}) Delta
// All four products run on MFMA.  The contraction order inside every 32-wide k
// step is permuted (kperm) so each accumulator is directly the next product's
// B operand.  fp32 operands (M0, R, Delta, T, P) are split into bf16 hi + lo;
// bf16 inputs (K, Q) are exact operands.
//
// The chunk's operands (K record, T, P, row scalars, V columns) are copied
// global -> LDS by DMA (global_load_lds, 16 bytes per lane) into one of two
// LDS buffers while the other buffer's chunk computes; every operand is then
// read with 16-byte LDS loads.
#pragma once

#include "gdn_device.h"
#include "gdn_intra.h"
#include "gdn_plan.h"

namespace gdn {

constexpr int kScanWaves = 2;
constexpr int kScanCols = 16 * kScanWaves;   // state columns per workgroup
constexpr int kLdsBytes = 160 * 1024;

typedef __attribute__((address_space(3))) void* lds_ptr_t;

// 16 bytes per lane from `src` (per lane) to LDS `dst + 16 * lane` (dst uniform).
__device__ __forceinline__ void dma16(const void* src, void* dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr_t)dst, 16, 0, 0);
}

__device__ __forceinline__ void wait_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// LDS layout of one chunk buffer.
template <typename TIn, int DK, bool FWD>
struct ScanLds {
  static constexpr bool kSplit = sizeof(TIn) == 4;
  static constexpr int kNL = kSplit ? 2 : 1;
  static constexpr int kKFrags = k_record_frags(DK, FWD);                  // per part
  static constexpr int kKBytes = static_cast<int>(k_record_bytes(DK, FWD, kSplit));
  static constexpr int kTBytes = static_cast<int>(kTRecordBytes);
  static constexpr int kPBytes = FWD ? static_cast<int>(kPRecordBytes) : 0;
  static constexpr int kSBytes = static_cast<int>(kSRecordBytes);
  static constexpr int kVBytes = kChunk * kScanCols * static_cast<int>(sizeof(TIn));
  static constexpr int kOffK = 0;
  static constexpr int kOffT = kOffK + kKBytes;
  static constexpr int kOffP = kOffT + kTBytes;
  static constexpr int kOffS = kOffP + kPBytes;
  static constexpr int kOffV = kOffS + kSBytes;
  static constexpr int kBytes = kOffV + kVBytes;
  static constexpr int kBuffers = 2 * kBytes <= kLdsBytes ? 2 : 1;
  // 1 KiB DMA blocks of fragments (K record, T, P): contiguous in LDS
  static constexpr int kFragBlocks = (kKBytes + kTBytes + kPBytes) / 1024;
  static constexpr int kVRowsPerBlock = 64 * 16 / (kScanCols * static_cast<int>(sizeof(TIn)));
  static constexpr int kVBlocks = kChunk / kVRowsPerBlock;
};

template <typename TIn, int DK, bool FWD>
__global__ __launch_bounds__(kScanWaves * kWave) __attribute__((amdgpu_waves_per_eu(1, 1)))
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
  __shared__ __attribute__((aligned(1024))) unsigned char lds[L::kBuffers * L::kBytes];

  const int tid = threadIdx.x;
  // wave index made provably uniform: DMA destinations (M0) stay scalar
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int lg = lane / 16, lr = lane % 16;
  const int ngroups = dv / kScanCols;
  const int unit = blockIdx.x;
  const int cgrp = unit % ngroups;
  const int h = (unit / ngroups) % hv;
  const int n = unit / (ngroups * hv);
  const int kh = h / (hv / hk);
  const int col0 = kScanCols * cgrp;           // first column of the workgroup
  const int wcol = 16 * wave + lr;             // this lane's column within the workgroup
  const int col = col0 + wcol;
  const int tok0 = cu[n];
  const int len = cu[n + 1] - tok0;
  const int slot0 = tok0 / kChunk + n;
  const int nch = (len + kChunk - 1) / kChunk;
  const int64_t vrow = static_cast<int64_t>(hv) * dv;   // token stride of v and o

  // ---- copy chunk ci's operands into LDS buffer b (both waves share the blocks)
  auto dma_chunk = [&](int ci, int b) __attribute__((always_inline)) {
    unsigned char* base = lds + b * L::kBytes;
    const int64_t srec = static_cast<int64_t>(slot0 + ci);
    const unsigned char* krec = reinterpret_cast<const unsigned char*>(Kw) + (srec * hk + kh) * L::kKBytes;
    const unsigned char* trec = reinterpret_cast<const unsigned char*>(Tw) + (srec * hv + h) * L::kTBytes;
    const unsigned char* prec = reinterpret_cast<const unsigned char*>(Pw) + (srec * hv + h) * L::kPBytes;
    for (int blk = wave; blk < L::kFragBlocks; blk += kScanWaves) {
      const int off = blk * 1024;
      const unsigned char* src = off < L::kKBytes ? krec + off
                               : off < L::kKBytes + L::kTBytes ? trec + (off - L::kKBytes)
                               : prec + (off - L::kKBytes - L::kTBytes);
      dma16(src + 16 * lane, base + off);
    }
    // row scalars: 1280 bytes = one full block and a quarter block
    const unsigned char* srow = reinterpret_cast<const unsigned char*>(Sw) + (srec * hv + h) * L::kSBytes;
    if (wave == 0) dma16(srow + 16 * lane, base + L::kOffS);
    else if (lane < 16) dma16(srow + 1024 + 16 * lane, base + L::kOffS + 1024);
    // V columns [col0, col0 + 32) of the chunk's rows; pad rows repeat the last
    // row (their beta is 0, so they contribute nothing)
    const int t0 = tok0 + ci * kChunk;
    const int clen = min(kChunk, len - ci * kChunk);
    constexpr int LPR = 64 / L::kVRowsPerBlock;              // lanes per row
    constexpr int EPL = 16 / static_cast<int>(sizeof(TIn));  // elements per lane
    for (int blk = wave; blk < L::kVBlocks; blk += kScanWaves) {
      const int i = min(blk * L::kVRowsPerBlock + lane / LPR, clen - 1);
      const TIn* src = v + static_cast<int64_t>(t0 + i) * vrow + static_cast<int64_t>(h) * dv + col0 +
                       (lane % LPR) * EPL;
      dma16(src, base + L::kOffV + blk * 1024);
    }
  };

  // state M, accumulator layout: M[td][r] = M[16 td + 4 lg + r][col]
  f32x4 M[NT];
  const int64_t sbase = (static_cast<int64_t>(n) * hv + h) * DK * dv + col;
  if (state_in != nullptr) {
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        M[td][r] = state_in[sbase + static_cast<int64_t>(16 * td + 4 * lg + r) * dv];
  } else {
#pragma unroll
    for (int td = 0; td < NT; ++td) M[td] = zero4();
  }

  if (nch > 0) {
    dma_chunk(0, 0);
    wait_dma();
    __syncthreads();
  }

  for (int ci = 0; ci < nch; ++ci) {
    const int b = L::kBuffers == 2 ? (ci & 1) : 0;
    if (L::kBuffers == 2 && ci + 1 < nch) dma_chunk(ci + 1, b ^ 1);   // in flight during compute

    const unsigned char* base = lds + b * L::kBytes;
    const u32x4* kf = reinterpret_cast<const u32x4*>(base + L::kOffK);
    const u32x4* tf = reinterpret_cast<const u32x4*>(base + L::kOffT);
    const u32x4* pf = reinterpret_cast<const u32x4*>(base + L::kOffP);
    const float* sc = reinterpret_cast<const float*>(base + L::kOffS);
    const TIn* vt = reinterpret_cast<const TIn*>(base + L::kOffV);
    const int t0 = tok0 + ci * kChunk;
    const int clen = min(kChunk, len - ci * kChunk);
    auto frag = [&](const u32x4* p, int f) __attribute__((always_inline)) {
      return __builtin_bit_cast(bf16x8, p[f * kWave + lane]);
    };

    // Operand fragments are loaded one phase ahead of the MFMAs that use them,
    // so LDS latency overlaps matrix work.
    bf16x8 ka[4][NK], kal[SPLIT ? 4 : 1][SPLIT ? NK : 1];
    bf16x8 qa[FWD ? 4 : 1][FWD ? NK : 1], qal[FWD && SPLIT ? 4 : 1][FWD && SPLIT ? NK : 1];
#pragma unroll
    for (int ti = 0; ti < 4; ++ti)
#pragma unroll
      for (int kk = 0; kk < NK; ++kk) {
        ka[ti][kk] = frag(kf, ti * NK + kk);
        if constexpr (SPLIT) kal[ti][kk] = frag(kf, L::kKFrags + ti * NK + kk);
        if constexpr (FWD) {
          qa[ti][kk] = frag(kf, NKA + NKT + ti * NK + kk);
          if constexpr (SPLIT) qal[ti][kk] = frag(kf, L::kKFrags + NKA + NKT + ti * NK + kk);
        }
      }
    Frag tfr[kTFrags];
#pragma unroll
    for (int f = 0; f < kTFrags; ++f) {
      tfr[f].hi = frag(tf, f);
      tfr[f].lo = frag(tf, kTFrags + f);
    }
    __builtin_amdgcn_sched_barrier(0);   // keep the loads ahead of the MFMAs

    // ---- K M0 and Q M0 (M0 split hi/lo as B operand)
    f32x4 km[4], qm[4];
#pragma unroll
    for (int ti = 0; ti < 4; ++ti) { km[ti] = zero4(); qm[ti] = zero4(); }
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      const Frag mb = chain_frag(M[2 * kk], M[2 * kk + 1]);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        Frag a;
        a.hi = ka[ti][kk];
        if constexpr (SPLIT) a.lo = kal[ti][kk];
        km[ti] = mma_a<SPLIT>(a, mb, km[ti]);
        if constexpr (FWD) {
          Frag aq;
          aq.hi = qa[ti][kk];
          if constexpr (SPLIT) aq.lo = qal[ti][kk];
          qm[ti] = mma_a<SPLIT>(aq, mb, qm[ti]);
        }
      }
    }

    // next phases' operands: K^T (and P)
    bf16x8 kt[NT][2], ktl[SPLIT ? NT : 1][2];
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        kt[td][kk] = frag(kf, NKA + 2 * td + kk);
        if constexpr (SPLIT) ktl[td][kk] = frag(kf, L::kKFrags + NKA + 2 * td + kk);
      }
    Frag pfr[FWD ? kTFrags : 1];
    if constexpr (FWD) {
#pragma unroll
      for (int f = 0; f < kTFrags; ++f) {
        pfr[f].hi = frag(pf, f);
        pfr[f].lo = frag(pf, kTFrags + f);
      }
    }
    __builtin_amdgcn_sched_barrier(0);

    // ---- R = beta V - beta e^G (K M0); rows 16 ti + 4 lg + r of this lane's column
    f32x4 R[4];
#pragma unroll
    for (int ti = 0; ti < 4; ++ti) {
      const int i0 = 16 * ti + 4 * lg;
      const f32x4 bta = *reinterpret_cast<const f32x4*>(sc + 0 * kChunk + i0);
      const f32x4 bge = *reinterpret_cast<const f32x4*>(sc + 1 * kChunk + i0);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float vv = load_elt(vt, (i0 + r) * kScanCols + wcol);
        R[ti][r] = bta[r] * vv - bge[r] * km[ti][r];
      }
    }

    // ---- Delta = T R (T lower triangular: k step 1 only for row tiles 2, 3)
    f32x4 D[4];
    {
      const Frag rb0 = chain_frag(R[0], R[1]);
      const Frag rb1 = chain_frag(R[2], R[3]);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        f32x4 acc = zero4();
#pragma unroll
        for (int kk = 0; kk <= ti / 2; ++kk) acc = mma_x3(tfr[tri_frag(ti, kk)], kk == 0 ? rb0 : rb1, acc);
        D[ti] = acc;
      }
    }

    // ---- outputs O = scale e^G (Q M0) + P Delta
    if constexpr (FWD) {
      const Frag db0 = chain_frag(D[0], D[1]);
      const Frag db1 = chain_frag(D[2], D[3]);
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        const int i0 = 16 * ti + 4 * lg;
        const f32x4 qe = *reinterpret_cast<const f32x4*>(sc + 3 * kChunk + i0);
        f32x4 acc;
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = qe[r] * qm[ti][r];
#pragma unroll
        for (int kk = 0; kk <= ti / 2; ++kk) acc = mma_x3(pfr[tri_frag(ti, kk)], kk == 0 ? db0 : db1, acc);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int i = i0 + r;
          if (i < clen) store_elt(o, (static_cast<int64_t>(t0 + i) * hv + h) * dv + col, acc[r]);
        }
      }
    }

    // ---- M1 = e^{G_last} M0 + K^T diag(e^{G_last - G}) Delta
    {
      f32x4 Dw[4];
#pragma unroll
      for (int ti = 0; ti < 4; ++ti) {
        const f32x4 w = *reinterpret_cast<const f32x4*>(sc + 2 * kChunk + 16 * ti + 4 * lg);
#pragma unroll
        for (int r = 0; r < 4; ++r) Dw[ti][r] = w[r] * D[ti][r];
      }
      const Frag db0 = chain_frag(Dw[0], Dw[1]);
      const Frag db1 = chain_frag(Dw[2], Dw[3]);
      const float eg = sc[4 * kChunk];
#pragma unroll
      for (int td = 0; td < NT; ++td) {
        f32x4 acc;
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[r] = eg * M[td][r];
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) {
          Frag a;
          a.hi = kt[td][kk];
          if constexpr (SPLIT) a.lo = ktl[td][kk];
          acc = mma_a<SPLIT>(a, kk == 0 ? db0 : db1, acc);
        }
        M[td] = acc;
      }
    }

    if (L::kBuffers == 1) {
      __syncthreads();   // everyone is done with the only buffer
      if (ci + 1 < nch) dma_chunk(ci + 1, 0);
    }
    wait_dma();
    __syncthreads();     // next chunk's operands are in LDS; this buffer is free
  }

  if (state_out) {
#pragma unroll
    for (int td = 0; td < NT; ++td)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        state_out[sbase + static_cast<int64_t>(16 * td + 4 * lg + r) * dv] = M[td][r];
  }
}

}  // namespace gdn
