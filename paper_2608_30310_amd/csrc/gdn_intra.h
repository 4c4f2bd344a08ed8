// Intra-chunk kernel: everything about one 64-token chunk that does not depend
// on the recurrent state, for one value head.
//
// For chunk rows i, j (0..63) with in-chunk inclusive cumulative log-gate G:
//   A_ij = beta_i e^{G_i - G_j} (k_i . k_j)   for j < i, else 0
//   T    = (I + A)^-1                          unit lower triangular
//   P_ij = scale e^{G_i - G_j} (q_i . k_j)     for j <= i, else 0   (outputs only)
// K K^T and Q K^T run on MFMA (bf16 inputs are exact operands; fp32 inputs are
// split hi/lo).  T is formed in fp32: the four diagonal 16x16 blocks by forward
// substitution in registers, then the off-diagonal blocks from the inverse of a
// 2x2 lower block triangular matrix (lower-left block -T22 A21 T11), applied to
// 16-row blocks and then to the 32-row halves, with fp32 MFMA (exact fp32
// products).
//
// Everything is written to the workspace as ready-made MFMA A operands in the
// order the scan consumes them (k slots permuted by kperm): T and P split into
// bf16 hi/lo (only their six nonzero fragments; T hi only for bf16 inputs), the
// per-row scalars and, by the first value head of each key head, the K record
// (K and Q as operands; split into hi/lo for fp32 inputs).
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

// LDS of one intra workgroup, which prepares HPW value heads of one key head
// (the key rows and K K^T are shared; outputs need P per head and keep one).
template <typename TIn, int DK, bool FWD, int HPW = 1>
struct IntraLds {
  static_assert(HPW == 1 || (HPW == 2 && !FWD), "two value heads per workgroup for tail replay only");
  static constexpr bool kSplit = sizeof(TIn) == 4;
  // Row pitches are an odd multiple of 32 bytes: 16-byte reads of 16
  // consecutive rows at one column (K K^T operands, record rows) are then
  // free of bank conflicts on gfx950, where pitches of 16 or 48 bytes past a
  // multiple of 64 cost 4 conflict cycles per read (measured with
  // SQ_LDS_BANK_CONFLICT).
  static constexpr int KP = DK + 16;                // padded LDS row (bf16 elements)
  static constexpr int NL = kSplit ? 2 : 1;         // hi (and lo) copies
  static constexpr int AP = kChunk + 8;             // fp32 row pitch of A, T and P
  // A takes the keys' place: every read of the key tile (the operands of
  // K K^T and of the K record) is issued and waited for before the first
  // element of A is written.  Likewise P takes the queries' place.  And
  // T = (I + A)^-1 is formed in A's place: every step of the inversion reads
  // the blocks of A it needs before it writes the T block that replaces one of
  // them, and never reads that A block again.  Sizes (bf16, d_k = 128): tail
  // replay of two value heads 37 KiB (four workgroups per CU), of one 18.5
  // KiB (eight), forward 36.5 KiB (four).
  union {
    alignas(16) uint16_t Ks[NL][kChunk][KP];
    alignas(16) float As[HPW][kChunk][AP];          // A (strictly lower), then T = (I + A)^-1
  };
  union {
    alignas(16) uint16_t Qs[FWD ? NL : 1][FWD ? kChunk : 1][KP];
    alignas(16) float Ps[FWD ? kChunk : 1][AP];
  };
  alignas(16) float Gs[HPW][kChunk];
  alignas(16) float Bs[HPW][kChunk];
};

// One intra workgroup for chunk slot `slot` and value heads h0 .. h0 + HPW - 1
// (of one key head), with its LDS in `sm`.  The work is laid out for four
// waves (256 threads); a workgroup launched with more leaves the extra waves
// idle except for the barriers.
template <typename TIn, int DK, bool FWD, int HPW = 1>
__device__ __forceinline__ void intra_body(IntraLds<TIn, DK, FWD, HPW>& sm, int slot, int h0,
                                           const int32_t* __restrict__ cu, int32_t num_seqs,
                                           int32_t hk, int32_t hv,
                                           const TIn* __restrict__ q,
                                           const TIn* __restrict__ k,
                                           const float* __restrict__ g,
                                           const float* __restrict__ beta, float scale,
                                           u32x4* __restrict__ Kw,
                                           u32x4* __restrict__ Tw,
                                           float* __restrict__ Sw,
                                           u32x4* __restrict__ Pw) {
  using S = IntraLds<TIn, DK, FWD, HPW>;
  constexpr bool SPLIT = S::kSplit;
  constexpr int KP = S::KP;
  constexpr int NL = S::NL;
  constexpr int AP = S::AP;
  constexpr int NK = DK / 32;
  constexpr int NKA = ka_frags(DK);
  constexpr int NKF = k_record_frags(DK, FWD);   // fragments per bf16 part
  auto& Ks = sm.Ks;
  auto& Qs = sm.Qs;
  auto& As = sm.As;
  auto& Ts = sm.As;   // T overwrites A block by block (see IntraLds)
  auto& Ps = sm.Ps;
  auto& Gs = sm.Gs;
  auto& Bs = sm.Bs;
  (void)KP;

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int lg = lane / 16, lr = lane % 16;
  const int grp = hv / hk;
  const int kh = h0 / grp;

  int seq, start, len;
  if (!slot_owner(cu, num_seqs, slot, seq, start, len)) return;   // uniform over the block

  constexpr int kWork = 4;   // waves that work
  // ---- all global loads first: K (and Q) rows, the heads' gates and betas
  //      (wave hh < HPW: value head h0 + hh)
  if (wave < kWork) {
    const int64_t off = (static_cast<int64_t>(start) * hk + kh) * DK;
    RowTile<TIn, DK> kt, qt;
    kt.load(k + off, static_cast<int64_t>(hk) * DK, len, tid);
    if constexpr (FWD) qt.load(q + off, static_cast<int64_t>(hk) * DK, len, tid);
    float gx = 0.f, bx = 0.f;
    if (wave < HPW) {
      const int64_t gi = static_cast<int64_t>(start + min(lane, len - 1)) * hv + h0 + wave;
      gx = g[gi];
      bx = beta[gi];
    }
    store_rows<TIn, DK, NL, KP>(Ks, kt, tid);
    if constexpr (FWD) store_rows<TIn, DK, NL, KP>(Qs, qt, tid);
    if (wave < HPW) {
      // inclusive cumulative log-gate; pad rows carry g = 0 and beta = 0
      float x = lane < len ? gx : 0.f;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const float y = __shfl_up(x, o, kWave);
        if (lane >= o) x += y;
      }
      Gs[wave][lane] = x;
      Bs[wave][lane] = lane < len ? bx : 0.f;
    }
  }
  __syncthreads();

  // ---- K K^T (and Q K^T) on MFMA, 10 lower tiles over 4 waves (tiles wave,
  //      wave + 4, wave + 8), and for fp32 inputs the K record of this key
  //      head (written by the workgroup of the group's first value head,
  //      waves 1..3; bf16 inputs need none: the scan fetches the key rows
  //      themselves).  Every read of the key (and query) tile happens before
  //      the barrier below, since A (and P) take their LDS afterwards; the
  //      MFMAs run before it too, so only the accumulators and the record
  //      fragments wait in registers.
  //      K record fragment f, lane (g, r), element j:
  //        K   (ti, kk): K[16 ti + r][32 kk + 8 g + j]                f = ti * NK + kk
  //        Q   (ti, kk): Q[16 ti + r][32 kk + 8 g + j]                f = NKA + ti * NK + kk
  //      record layout [hi | lo][fragment][kslot(lane)]
  constexpr int TPW = 3;   // tiles of K K^T per wave, at most
  constexpr int PA = (NKA + 2) / 3;   // K record fragments per writer wave, per part
  const bool writer = SPLIT && wave >= 1 && wave < kWork && h0 % grp == 0;
  const int w3 = wave - 1;             // writer index 0..2
  f32x4 acc[TPW], accq[TPW];
  u32x4 va[NL][PA], vq[FWD ? NL : 1][FWD ? PA : 1];
  auto tile_rc = [](int t, int& bi, int& bj) __attribute__((always_inline)) {
    bi = t < 1 ? 0 : t < 3 ? 1 : t < 6 ? 2 : 3;
    bj = t - bi * (bi + 1) / 2;
  };
  if (wave < kWork) {
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      acc[u] = zero4();
      accq[u] = zero4();
      const int t = wave + 4 * u;
      if (t < 10) {
        int bi, bj;
        tile_rc(t, bi, bj);
#pragma unroll
        for (int kk = 0; kk < NK; ++kk) {
          const int c = 32 * kk + 8 * lg;
          Frag fa, fb, fq;
          fa.hi = *reinterpret_cast<const bf16x8*>(&Ks[0][16 * bi + lr][c]);
          fb.hi = *reinterpret_cast<const bf16x8*>(&Ks[0][16 * bj + lr][c]);
          if constexpr (SPLIT) {
            fa.lo = *reinterpret_cast<const bf16x8*>(&Ks[NL - 1][16 * bi + lr][c]);
            fb.lo = *reinterpret_cast<const bf16x8*>(&Ks[NL - 1][16 * bj + lr][c]);
          }
          if constexpr (FWD) {
            fq.hi = *reinterpret_cast<const bf16x8*>(&Qs[0][16 * bi + lr][c]);
            if constexpr (SPLIT) fq.lo = *reinterpret_cast<const bf16x8*>(&Qs[NL - 1][16 * bi + lr][c]);
          }
          if constexpr (SPLIT) {
            acc[u] = mma_x3(fa, fb, acc[u]);
            if constexpr (FWD) accq[u] = mma_x3(fq, fb, accq[u]);
          } else {
            acc[u] = mma(fa.hi, fb.hi, acc[u]);
            if constexpr (FWD) accq[u] = mma(fq.hi, fb.hi, accq[u]);
          }
        }
      }
    }
    if (writer) {
      // fragment indices clamped so the reads are unconditional
#pragma unroll
      for (int p = 0; p < NL; ++p)
#pragma unroll
        for (int i = 0; i < PA; ++i) {
          const int f = min(w3 + 3 * i, NKA - 1);
          const int ti = f / NK, kk = f % NK;
          va[p][i] = *reinterpret_cast<const u32x4*>(&Ks[p][16 * ti + lr][32 * kk + 8 * lg]);
          if constexpr (FWD) vq[p][i] = *reinterpret_cast<const u32x4*>(&Qs[p][16 * ti + lr][32 * kk + 8 * lg]);
        }
    }
  }
  __syncthreads();   // the key and query tiles are dead from here

  if (wave < kWork) {
    // A (and P) of every head from the shared accumulators
#pragma unroll
    for (int u = 0; u < TPW; ++u) {
      const int t = wave + 4 * u;
      if (t < 10) {
        int bi, bj;
        tile_rc(t, bi, bj);
        const int j = 16 * bj + lr;
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
          const float gj = Gs[hh][j];
          const f32x4 gi = *reinterpret_cast<const f32x4*>(&Gs[hh][16 * bi + 4 * lg]);
          const f32x4 bi4 = *reinterpret_cast<const f32x4*>(&Bs[hh][16 * bi + 4 * lg]);
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int i = 16 * bi + 4 * lg + r;
            const float decay = j <= i ? __expf(gi[r] - gj) : 0.f;
            As[hh][i][j] = j < i ? bi4[r] * decay * acc[u][r] : 0.f;
            if constexpr (FWD) Ps[i][j] = scale * decay * accq[u][r];
          }
        }
      }
    }
    if (writer) {
      u32x4* kdst = Kw + (static_cast<int64_t>(slot) * hk + kh) * (NL * NKF * kWave);
#pragma unroll
      for (int p = 0; p < NL; ++p) {
        u32x4* pdst = kdst + static_cast<int64_t>(p) * NKF * kWave;
#pragma unroll
        for (int i = 0; i < PA; ++i) {
          const int f = w3 + 3 * i;
          if (f < NKA) {
            pdst[f * kWave + kslot(lane)] = va[p][i];
            if constexpr (FWD) pdst[(NKA + f) * kWave + kslot(lane)] = vq[p][i];
          }
        }
      }
    }
  }
  __syncthreads();

  if (wave < HPW) {
    // ---- diagonal 16x16 blocks of T of head `wave`: lane = (block b, column
    //      j).  The block's rows are read once as 16-byte pieces; forward
    //      substitution runs right-looking (row i takes A_im x_m as soon as x_m
    //      is final), so every step has independent FMAs.
    auto& A = As[wave];
    const int b = lane >> 4, jj = lane & 15;
    f32x4 arow[16][4];
#pragma unroll
    for (int i = 1; i < 16; ++i)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        if (4 * c < i) arow[i][c] = *reinterpret_cast<const f32x4*>(&A[16 * b + i][16 * b + 4 * c]);
    float x[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) x[i] = (i == jj) ? 1.f : 0.f;
#pragma unroll
    for (int m = 0; m < 15; ++m)
#pragma unroll
      for (int i = m + 1; i < 16; ++i) x[i] -= arow[i][m / 4][m % 4] * x[m];
#pragma unroll
    for (int i = 0; i < 16; ++i) A[16 * b + i][16 * b + jj] = x[i];
  } else if (wave < 2 * HPW) {
    // ---- meanwhile, the per-row scalars of head `wave - HPW` for the scan
    const int hh = wave - HPW;
    const float gl = Gs[hh][kChunk - 1];   // pad rows carry g = 0, so this is the last token's G
    float* sc = Sw + (static_cast<int64_t>(slot) * hv + h0 + hh) * (kScalarRows * kChunk);
    sc[0 * kChunk + lane] = Bs[hh][lane];
    sc[1 * kChunk + lane] = Bs[hh][lane] * __expf(Gs[hh][lane]);
    sc[2 * kChunk + lane] = __expf(gl - Gs[hh][lane]);
    sc[3 * kChunk + lane] = scale * __expf(Gs[hh][lane]);
    sc[4 * kChunk + lane] = __expf(gl);
  }
  __syncthreads();

  // ---- off-diagonal blocks by the block-inverse identity for a lower block
  //      triangular matrix: inv([[I + A11, 0], [A21, I + A22]]) has lower-left
  //      block -T22 A21 T11.  First on 16-row blocks (T_10, T_32), then on the
  //      32-row halves (rows 32..63, columns 0..31).  fp32 MFMA throughout.
  //      blk_mm: acc += X[16 x 16] Y[16 x 16], both in LDS (row pitches xp,
  //      yp), contraction index 4 kk + (lane / 16) in k step kk.
  auto blk_mm = [&](f32x4 acc, const float* X, int xp, const float* Y, int yp) __attribute__((always_inline)) {
    float xa[4], yb[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      xa[kk] = X[lr * xp + 4 * kk + lg];
      yb[kk] = Y[(4 * kk + lg) * yp + lr];
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc = mma_f32(xa[kk], yb[kk], acc);
    return acc;
  };
  //      blk_mm_reg: acc += X[16 x 16] (LDS) Y, Y the accumulator of an
  //      earlier product (lane (g, c) holds Y[4 g + i][c]): with contraction
  //      index 4 (lane / 16) + kk in k step kk, B is the lane's own y[kk].
  auto blk_mm_reg = [&](f32x4 acc, const float* X, int xp, const f32x4& y) __attribute__((always_inline)) {
    float xa[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) xa[kk] = X[lr * xp + 4 * lg + kk];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) acc = mma_f32(xa[kk], y[kk], acc);
    return acc;
  };
  auto at = [&](float (*M)[AP], int r, int c) __attribute__((always_inline)) { return &M[16 * r][16 * c]; };
  if (wave < 2 * HPW) {
    // T_ab = -T_aa A_ab T_bb for (a, b) = (1, 0) and (3, 2) of head wave / 2;
    // A_ab is read by this wave alone, so T_ab takes its place directly
    auto& T = Ts[wave / 2];
    const int a = 2 * (wave % 2) + 1, bb = a - 1;
    const f32x4 y = blk_mm(zero4(), at(T, a, bb), AP, at(T, bb, bb), AP);
    const f32x4 xx = blk_mm_reg(zero4(), at(T, a, a), AP, y);
#pragma unroll
    for (int r = 0; r < 4; ++r) T[16 * a + 4 * lg + r][16 * bb + lr] = -xx[r];
  }
  __syncthreads();
  // rows 32..63, columns 0..31, block (rr, cc) of each head: Y_k = A[k, 0:32]
  // T[0:32, cc] for row blocks k = 2 .. rr (T_jc = 0 for j < c), then
  // -sum_k T_rr,k Y_k; the Y of a block are recomputed by every block that
  // needs them, so they stay in registers.  Blocks by cost 12, 8, 24, 16
  // MFMAs: wave w takes block w of head 0 and block 3 - w of head 1.
  f32x4 xo[HPW];
  if (wave < kWork) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      auto& T = Ts[hh];
      const int blk = hh == 0 ? wave : 3 - wave;
      const int rr = 2 + blk / 2, cc = blk % 2;
      f32x4 yk[2];
#pragma unroll
      for (int kr = 2; kr < 4; ++kr) {
        if (kr > rr) break;
        f32x4 y = zero4();
#pragma unroll
        for (int j = 0; j < 2; ++j)
          if (j >= cc) y = blk_mm(y, at(T, kr, j), AP, at(T, j, cc), AP);
        yk[kr - 2] = y;
      }
      f32x4 xx = zero4();
#pragma unroll
      for (int kr = 2; kr < 4; ++kr)
        if (kr <= rr) xx = blk_mm_reg(xx, at(T, rr, kr), AP, yk[kr - 2]);
      xo[hh] = xx;
    }
  }
  __syncthreads();   // every read of the lower-left blocks of A is done
  if (wave < kWork) {
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
      const int blk = hh == 0 ? wave : 3 - wave;
      const int rr = 2 + blk / 2, cc = blk % 2;
#pragma unroll
      for (int r = 0; r < 4; ++r) Ts[hh][16 * rr + 4 * lg + r][16 * cc + lr] = -xo[hh][r];
    }
  }
  __syncthreads();

  // ---- T (and P) as split A fragments, nonzero ones only: fragment
  //      tri_frag(ti, kk), lane (g, r), element j = [16 ti + r][32 kk + kperm(g, j)];
  //      record layout [hi | lo][fragment][lane]; for bf16 inputs T keeps hi only
  constexpr int TPARTS = t_record_parts(SPLIT);
  constexpr int kRec = kTFrags * kWave;   // record entries per head
  for (int e2 = tid; wave < kWork && e2 < HPW * kRec; e2 += kWork * kWave) {
    const int hh = e2 / kRec, e = e2 % kRec;
    const int64_t rec = static_cast<int64_t>(slot) * hv + h0 + hh;
    const int f = e / kWave, fl = e % kWave;
    const int ti = f < 2 ? f : 2 + (f - 2) / 2, kk = f < 2 ? 0 : (f - 2) % 2;
    const int fg = fl / 16, fr = fl % 16;
    const int row = 16 * ti + fr;
    // the lane's elements j < 4 are columns 32 kk + 4 fg .. + 3 (column block
    // 2 kk) and j >= 4 the same 16 columns further (block 2 kk + 1): two
    // 16-byte reads, conflict-free (rows 72 floats apart);
    // blocks above the diagonal are zero
    const int c0 = 32 * kk + 4 * fg;
    const bool lo_blk = 2 * kk <= ti, hi_blk = 2 * kk + 1 <= ti;
    const f32x4 t0 = lo_blk ? *reinterpret_cast<const f32x4*>(&Ts[hh][row][c0]) : zero4();
    const f32x4 t1 = hi_blk ? *reinterpret_cast<const f32x4*>(&Ts[hh][row][c0 + 16]) : zero4();
    const float tv[8] = {t0[0], t0[1], t0[2], t0[3], t1[0], t1[1], t1[2], t1[3]};
    const Frag tf = split8(tv);
    u32x4* tdst = Tw + rec * (TPARTS * kRec);
    tdst[e] = __builtin_bit_cast(u32x4, tf.hi);
    if constexpr (TPARTS == 2) tdst[kRec + e] = __builtin_bit_cast(u32x4, tf.lo);
    if constexpr (FWD) {
      const f32x4 p0 = lo_blk ? *reinterpret_cast<const f32x4*>(&Ps[row][c0]) : zero4();
      const f32x4 p1 = hi_blk ? *reinterpret_cast<const f32x4*>(&Ps[row][c0 + 16]) : zero4();
      const float pv[8] = {p0[0], p0[1], p0[2], p0[3], p1[0], p1[1], p1[2], p1[3]};
      const Frag pf = split8(pv);
      u32x4* pdst = Pw + rec * (2 * kRec);
      pdst[e] = __builtin_bit_cast(u32x4, pf.hi);
      pdst[kRec + e] = __builtin_bit_cast(u32x4, pf.lo);
    }
  }
}

// Logical (slot, first value head) of intra workgroup i of n = slots x Hv /
// HPW: the value heads of one key head read the same key rows, so their
// workgroups form one cluster on one XCD (the second finds the rows in that
// XCD's L2), consecutive clusters on consecutive XCDs.  A bijection, so
// correctness does not depend on it.
template <int HPW = 1>
__device__ __forceinline__ void intra_unit(int i, int n, int hv, int grp, int& slot, int& h0) {
  const int u = xcd_cluster_remap(i, n, grp / HPW);
  slot = u / (hv / HPW);
  h0 = (u % (hv / HPW)) * HPW;
}

// grid = (num_slots, Hv / HPW): one workgroup per (chunk slot, HPW value heads
// of one key head).
template <typename TIn, int DK, bool FWD, int HPW = 1>
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
  __shared__ IntraLds<TIn, DK, FWD, HPW> sm;
  int slot, h0;
  intra_unit<HPW>(blockIdx.x + blockIdx.y * gridDim.x, gridDim.x * gridDim.y, hv, hv / hk, slot, h0);
  intra_body<TIn, DK, FWD, HPW>(sm, slot, h0, cu, num_seqs, hk, hv, q, k, g, beta, scale, Kw, Tw, Sw, Pw);
}

}  // namespace gdn
