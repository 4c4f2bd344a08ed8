// Intra-chunk kernel: everything about one 64-token chunk that does not depend
// on the recurrent state, for one value head.
//
// For chunk rows i, j (0..63) with in-chunk inclusive cumulative log-gate G:
//   A_ij = beta_i e^{G_i - G_j} (k_i . k_j)   for j < i, else 0
//   T    = (I + A)^-1                          unit lower triangular
//   P_ij = scale e^{G_i - G_j} (q_i . k_j)     for j <= i, else 0   (outputs only)
// K K^T and Q K^T run on MFMA (bf16 inputs are exact operands; fp32 inputs are
// split hi/lo).  T is formed in fp32 by blocked forward substitution: the four
// diagonal 16x16 blocks by column substitution in registers, then each column
// block b on its own wave, T_ab = -T_aa (sum_{m=b}^{a-1} A_am T_mb) for
// a = b+1..3, with fp32 MFMA (exact fp32 products).
//
// Everything is written to the workspace as ready-made MFMA A operands in the
// order the scan consumes them (k slots permuted by kperm): T and P split into
// bf16 hi/lo (only their six nonzero fragments), the per-row scalars and, by
// the first value head of each key head, the K record (K, K^T and Q as
// operands; split into hi/lo for fp32 inputs).
#pragma once

#include "gdn_device.h"
#include "gdn_plan.h"

namespace gdn {

constexpr int kScalarRows = 5;   // beta, beta e^G, e^{Gl-G}, scale e^G, e^{Gl}

// Nonzero fragments of a lower-triangular 64x64 operand: (row tile ti, k step kk)
// with kk <= ti / 2.
__device__ __forceinline__ int tri_frag(int ti, int kk) { return ti < 2 ? ti : 2 + 2 * (ti - 2) + kk; }

// Sequence and chunk of a workspace slot: slot(n, j) = cu[n]/64 + n + j is
// injective over all (sequence, chunk) pairs and needs no prefix sums.
__device__ __forceinline__ bool slot_owner(const int32_t* __restrict__ cu, int32_t num_seqs, int slot,
                                           int& seq, int& start, int& len) {
  int lo = 0, hi = num_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cu[mid] / kChunk + mid <= slot) lo = mid;
    else hi = mid - 1;
  }
  const int j = slot - (cu[lo] / kChunk + lo);
  const int slen = cu[lo + 1] - cu[lo];
  if (j < 0 || j * kChunk >= slen) return false;
  seq = lo;
  start = cu[lo] + j * kChunk;
  len = min(kChunk, slen - j * kChunk);
  return true;
}

// fp32 MFMA: D(16x16) += A(16x4) B(4x16).  Lane l supplies A[l%16][l/16] and
// B[l/16][l%16] and holds D[4(l/16)+i][l%16].
__device__ __forceinline__ f32x4 mma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// grid = (num_slots, Hv): one workgroup per (chunk slot, value head).
template <typename TIn, int DK, bool FWD>
__global__ __launch_bounds__(256) void k_intra(const int32_t* __restrict__ cu, int32_t num_seqs,
                                               int32_t hk, int32_t hv,
                                               const TIn* __restrict__ q,
                                               const TIn* __restrict__ k,
                                               const float* __restrict__ g,
                                               const float* __restrict__ beta, float scale,
                                               u32x4* __restrict__ Kw,
                                               u32x4* __restrict__ Tw,
                                               float* __restrict__ Sw,
                                               u32x4* __restrict__ Pw) {
  constexpr bool SPLIT = sizeof(TIn) == 4;   // fp32 inputs are not exact bf16
  constexpr int KP = DK + 8;                 // padded LDS row (bf16 elements)
  constexpr int NL = SPLIT ? 2 : 1;          // hi (and lo) copies
  constexpr int AP = kChunk + 4;             // fp32 row pitch of A, T and P
  constexpr int NK = DK / 32;
  constexpr int NKA = ka_frags(DK), NKT = kt_frags(DK);
  constexpr int NKF = k_record_frags(DK, FWD);   // fragments per bf16 part
  __shared__ __attribute__((aligned(16))) uint16_t Ks[NL][kChunk][KP];
  __shared__ __attribute__((aligned(16))) uint16_t Qs[FWD ? NL : 1][FWD ? kChunk : 1][KP];
  __shared__ __attribute__((aligned(16))) float As[kChunk][AP];   // A (strictly lower)
  __shared__ __attribute__((aligned(16))) float Ts[kChunk][AP];   // T = (I + A)^-1
  __shared__ __attribute__((aligned(16))) float Ps[FWD ? kChunk : 1][AP];
  __shared__ __attribute__((aligned(16))) float Ys[3][16][17];    // per-wave block scratch
  __shared__ float Gs[kChunk], Bs[kChunk];

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int lg = lane / 16, lr = lane % 16;
  const int slot = blockIdx.x;
  const int h = blockIdx.y;
  const int grp = hv / hk;
  const int kh = h / grp;
  const int64_t rec = static_cast<int64_t>(slot) * hv + h;

  int seq, start, len;
  if (!slot_owner(cu, num_seqs, slot, seq, start, len)) return;   // uniform over the block

  // ---- all global loads first: K (and Q) rows, this head's gates and betas
  {
    const int64_t off = (static_cast<int64_t>(start) * hk + kh) * DK;
    RowTile<TIn, DK> kt, qt;
    kt.load(k + off, static_cast<int64_t>(hk) * DK, len, tid);
    if constexpr (FWD) qt.load(q + off, static_cast<int64_t>(hk) * DK, len, tid);
    float gx = 0.f, bx = 0.f;
    if (wave == 0) {
      const int64_t gi = static_cast<int64_t>(start + min(lane, len - 1)) * hv + h;
      gx = g[gi];
      bx = beta[gi];
    }
    store_rows<TIn, DK, NL, KP>(Ks, kt, tid);
    if constexpr (FWD) store_rows<TIn, DK, NL, KP>(Qs, qt, tid);
    if (wave == 0) {
      // inclusive cumulative log-gate; pad rows carry g = 0 and beta = 0
      float x = lane < len ? gx : 0.f;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const float y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
      }
      Gs[lane] = x;
      Bs[lane] = lane < len ? bx : 0.f;
    }
  }
  __syncthreads();

  // ---- K K^T (and Q K^T) on MFMA, 10 lower tiles over 4 waves, turned into A (and P)
  for (int t = wave; t < 10; t += 4) {
    const int bi = t < 1 ? 0 : t < 3 ? 1 : t < 6 ? 2 : 3;
    const int bj = t - bi * (bi + 1) / 2;
    f32x4 acc = zero4(), accq = zero4();
#pragma unroll
    for (int kk = 0; kk < NK; ++kk) {
      const int c = 32 * kk + 8 * lg;
      Frag a, b;
      a.hi = *reinterpret_cast<const bf16x8*>(&Ks[0][16 * bi + lr][c]);
      b.hi = *reinterpret_cast<const bf16x8*>(&Ks[0][16 * bj + lr][c]);
      if constexpr (SPLIT) {
        a.lo = *reinterpret_cast<const bf16x8*>(&Ks[NL - 1][16 * bi + lr][c]);
        b.lo = *reinterpret_cast<const bf16x8*>(&Ks[NL - 1][16 * bj + lr][c]);
        acc = mma_x3(a, b, acc);
      } else {
        acc = mma(a.hi, b.hi, acc);
      }
      if constexpr (FWD) {
        Frag qa;
        qa.hi = *reinterpret_cast<const bf16x8*>(&Qs[0][16 * bi + lr][c]);
        if constexpr (SPLIT) {
          qa.lo = *reinterpret_cast<const bf16x8*>(&Qs[NL - 1][16 * bi + lr][c]);
          accq = mma_x3(qa, b, accq);
        } else {
          accq = mma(qa.hi, b.hi, accq);
        }
      }
    }
    const int j = 16 * bj + lr;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = 16 * bi + 4 * lg + r;
      const float decay = j <= i ? __expf(Gs[i] - Gs[j]) : 0.f;
      As[i][j] = j < i ? Bs[i] * decay * acc[r] : 0.f;
      if constexpr (FWD) Ps[i][j] = scale * decay * accq[r];
    }
  }
  __syncthreads();

  if (wave == 0) {
    // ---- diagonal 16x16 blocks of T: lane = (block, column), column substitution
    const int b = lane >> 4, jj = lane & 15;
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float s = (i == jj) ? 1.f : 0.f;
#pragma unroll
      for (int m = 0; m < i; ++m) s -= As[16 * b + i][16 * b + m] * x[m];
      x[i] = s;
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) Ts[16 * b + i][16 * b + jj] = x[i];
  } else if (h % grp == 0) {
    // ---- meanwhile, the K record of this key head: K, K^T (and Q) as bf16 A
    //      operands (hi and lo parts for fp32 inputs).
    //      fragment f, lane (g, r), element j:
    //        K   (ti, kk): K[16 ti + r][32 kk + kperm(g, j)]            f = ti * NK + kk
    //        K^T (td, kk): K[32 kk + kperm(g, j)][16 td + r]            f = NKA + 2 td + kk
    //        Q   (ti, kk): Q[16 ti + r][32 kk + kperm(g, j)]            f = NKA + NKT + ti * NK + kk
    //      record layout [hi | lo][fragment][lane]
    u32x4* kdst = Kw + (static_cast<int64_t>(slot) * hk + kh) * (NL * NKF * kWave);
    for (int e = tid - kWave; e < NL * NKF * kWave; e += 256 - kWave) {
      const int p = e / (NKF * kWave), f = (e / kWave) % NKF, fl = e % kWave;
      const int fg = fl / 16, fr = fl % 16;
      u32x4 val;
      if (f < NKA) {
        const int ti = f / NK, kk = f % NK;
        val = __builtin_bit_cast(u32x4, perm_frag(&Ks[p][16 * ti + fr][32 * kk + 4 * fg]));
      } else if (f < NKA + NKT) {
        const int td = (f - NKA) / 2, kk = (f - NKA) % 2;
        uint16_t v8[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v8[j] = Ks[p][32 * kk + kperm(fg, j)][16 * td + fr];
        val = u32x4{v8[0] | (uint32_t(v8[1]) << 16), v8[2] | (uint32_t(v8[3]) << 16),
                    v8[4] | (uint32_t(v8[5]) << 16), v8[6] | (uint32_t(v8[7]) << 16)};
      } else {
        const int fq = f - NKA - NKT;
        const int ti = fq / NK, kk = fq % NK;
        val = __builtin_bit_cast(
            u32x4, perm_frag(&Qs[FWD ? p : 0][FWD ? 16 * ti + fr : 0][FWD ? 32 * kk + 4 * fg : 0]));
      }
      kdst[e] = val;
    }
  }
  __syncthreads();

  // ---- off-diagonal blocks, one column block per wave (fp32 MFMA):
  //      T_ab = -T_aa (sum_{m=b}^{a-1} A_am T_mb), a = b+1..3
  if (wave < 3) {
    const int b = wave;
    for (int a = b + 1; a < 4; ++a) {
      f32x4 y = zero4();
      for (int m = b; m < a; ++m) {
#pragma unroll
        for (int kk = 0; kk < 4; ++kk)
          y = mma_f32(As[16 * a + lr][16 * m + 4 * kk + lg], Ts[16 * m + 4 * kk + lg][16 * b + lr], y);
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) Ys[b][4 * lg + r][lr] = y[r];
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
      f32x4 x = zero4();
#pragma unroll
      for (int kk = 0; kk < 4; ++kk)
        x = mma_f32(Ts[16 * a + lr][16 * a + 4 * kk + lg], Ys[b][4 * kk + lg][lr], x);
#pragma unroll
      for (int r = 0; r < 4; ++r) Ts[16 * a + 4 * lg + r][16 * b + lr] = -x[r];
      __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    }
  }
  __syncthreads();

  // ---- T (and P) as split A fragments, nonzero ones only: fragment
  //      tri_frag(ti, kk), lane (g, r), element j = [16 ti + r][32 kk + kperm(g, j)];
  //      record layout [hi | lo][fragment][lane]
  u32x4* tdst = Tw + rec * (2 * kTFrags * kWave);
  u32x4* pdst = FWD ? Pw + rec * (2 * kTFrags * kWave) : nullptr;
  for (int e = tid; e < kTFrags * kWave; e += 256) {
    const int f = e / kWave, fl = e % kWave;
    const int ti = f < 2 ? f : 2 + (f - 2) / 2, kk = f < 2 ? 0 : (f - 2) % 2;
    const int fg = fl / 16, fr = fl % 16;
    const int row = 16 * ti + fr;
    float tv[8], pv[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int col = 32 * kk + kperm(fg, j);
      const bool lower = col / 16 <= row / 16;
      tv[j] = lower ? Ts[row][col] : 0.f;
      if constexpr (FWD) pv[j] = lower ? Ps[row][col] : 0.f;
    }
    const Frag tf = split8(tv);
    tdst[e] = __builtin_bit_cast(u32x4, tf.hi);
    tdst[kTFrags * kWave + e] = __builtin_bit_cast(u32x4, tf.lo);
    if constexpr (FWD) {
      const Frag pf = split8(pv);
      pdst[e] = __builtin_bit_cast(u32x4, pf.hi);
      pdst[kTFrags * kWave + e] = __builtin_bit_cast(u32x4, pf.lo);
    }
  }
  // ---- per-row scalars for the scan
  if (tid < kChunk) {
    const float gl = Gs[kChunk - 1];   // pad rows carry g = 0, so this is the last token's G
    float* sc = Sw + rec * (kScalarRows * kChunk);
    sc[0 * kChunk + tid] = Bs[tid];
    sc[1 * kChunk + tid] = Bs[tid] * __expf(Gs[tid]);
    sc[2 * kChunk + tid] = __expf(gl - Gs[tid]);
    sc[3 * kChunk + tid] = scale * __expf(Gs[tid]);
    sc[4 * kChunk + tid] = __expf(gl);
  }
}

}  // namespace gdn
