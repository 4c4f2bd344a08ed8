// Decode-step kernel: one new token per sequence applied to a given state
// (paper Section 2, Eq. 1 for a single step; the first tokens generated after
// a prefix state has been rebuilt, Section 3).  With M = S^T and
// alpha = e^g, per (sequence, value head):
//   u  = M^T k                       (d_v)
//   d  = beta (v - alpha u)
//   M1 = alpha M + k d^T
//   o  = scale M1^T q
// The state is read once and written once, so the step is bound by HBM
// bandwidth: 2 d_k d_v fp32 values per (sequence, head) against a handful of
// flops each.  Both go through streaming (non-temporal) accesses: in a model,
// a layer's state comes back only after every other layer's, so keeping it in
// the caches gains nothing and evicts what does get reused.  Plain fp32 vector arithmetic; no MFMA (each state element takes
// part in two dot products of length d_k, too little work per byte for the
// matrix cores to matter).
//
// One workgroup (256 threads) per (sequence, value head): thread t owns the
// four columns 4 (t % (d_v / 4)).. of row part t / (d_v / 4), loaded as
// 16-byte vectors, so each load of a wave covers whole rows of the state
// (512 or 256 contiguous bytes).  The two dot products over d_k are reduced
// over the row parts with lane exchanges inside a wave and an LDS step across
// the eight waves.
#pragma once

#include "gdn_device.h"

namespace gdn {

constexpr int kDecodeThreads = 256;
constexpr int kDecodeWaves = kDecodeThreads / kWave;

// N consecutive elements (bf16 or fp32) from `p` as float, with the widest
// loads the run's size allows (the run starts at a multiple of its own size).
template <typename TIn, int N>
__device__ __forceinline__ void load_run(const TIn* __restrict__ p, float (&x)[N]) {
  constexpr int E = static_cast<int>(sizeof(TIn));
  constexpr int B = N * E;
  if constexpr (B % 16 == 0) {
#pragma unroll
    for (int j = 0; j < B / 16; ++j) {
      const u32x4 w = reinterpret_cast<const u32x4*>(p)[j];
#pragma unroll
      for (int e = 0; e < 16 / E; ++e) x[j * (16 / E) + e] = vec_elt<TIn>(w, e);
    }
  } else if constexpr (B == 8) {
    const u32x2 w = *reinterpret_cast<const u32x2*>(p);
#pragma unroll
    for (int e = 0; e < N; ++e) x[e] = vec_elt<TIn>(u32x4{w.x, w.y, 0u, 0u}, e);
  } else {
#pragma unroll
    for (int e = 0; e < N; ++e) x[e] = load_elt(p, e);
  }
}

// Sum over the row parts of the workgroup of a per-thread f32x4 (CQ column
// quads, lanes cq + CQ j of each wave); every thread receives the total for
// its column quad.  `red` is a kDecodeWaves x CQ LDS array.
template <int CQ>
__device__ __forceinline__ f32x4 decode_reduce(f32x4 x, f32x4 (*red)[CQ], int lane, int wave, int cq) {
#pragma unroll
  for (int off = CQ; off < kWave; off <<= 1)
#pragma unroll
    for (int c = 0; c < 4; ++c) x[c] += __shfl_xor(x[c], off, kWave);
  if (lane < CQ) red[wave][lane] = x;   // lane == cq here
  __syncthreads();
  f32x4 t = red[0][cq];
#pragma unroll
  for (int w = 1; w < kDecodeWaves; ++w)
#pragma unroll
    for (int c = 0; c < 4; ++c) t[c] += red[w][cq][c];
  return t;
}

// grid = N x Hv.  state_in NULL = zero state; state_out may equal state_in
// (each workgroup reads its whole slice before writing it).
template <typename TIn, int DK, int DV>
__global__ __launch_bounds__(kDecodeThreads)
void k_decode(int32_t hk, int32_t hv, const TIn* __restrict__ q, const TIn* __restrict__ k,
              const TIn* __restrict__ v, const float* __restrict__ g, const float* __restrict__ beta,
              float scale, const float* state_in, TIn* __restrict__ o, float* state_out) {
  constexpr int CQ = DV / 4;                  // column quads
  constexpr int RP = kDecodeThreads / CQ;     // row parts
  constexpr int RPT = DK / RP;                // rows per thread
  static_assert(RP * CQ == kDecodeThreads && RPT * RP == DK && kWave % CQ == 0, "decode tiling");
  __shared__ f32x4 red_u[kDecodeWaves][CQ], red_o[kDecodeWaves][CQ];
  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int lane = tid % kWave;
  const int cq = tid % CQ, rp = tid / CQ;
  const int unit = blockIdx.x;
  const int h = unit % hv, n = unit / hv;
  const int kh = h / (hv / hk);
  const int col = 4 * cq;
  const int64_t nh = static_cast<int64_t>(n) * hv + h;
  const int64_t sbase = nh * DK * DV + col;
  const int64_t kq = (static_cast<int64_t>(n) * hk + kh) * DK + rp * RPT;

  f32x4 m[RPT];
  if (state_in) {
#pragma unroll
    for (int i = 0; i < RPT; ++i)
      m[i] = __builtin_nontemporal_load(
          reinterpret_cast<const f32x4*>(state_in + sbase + static_cast<int64_t>(rp * RPT + i) * DV));
  } else {
#pragma unroll
    for (int i = 0; i < RPT; ++i) m[i] = zero4();
  }
  float kx[RPT], qx[RPT], vx[4];
  load_run<TIn, RPT>(k + kq, kx);
  load_run<TIn, RPT>(q + kq, qx);
  load_run<TIn, 4>(v + nh * DV + col, vx);
  const float alpha = __expf(g[nh]), b = beta[nh];

  // u = M^T k over this thread's rows, then over all rows
  f32x4 s = zero4();
#pragma unroll
  for (int i = 0; i < RPT; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) s[c] = fmaf(kx[i], m[i][c], s[c]);
  const f32x4 u = decode_reduce<CQ>(s, red_u, lane, wave, cq);

  // d = beta (v - alpha u); M1 = alpha M + k d^T; partial o = M1^T q
  f32x4 d, p = zero4();
#pragma unroll
  for (int c = 0; c < 4; ++c) d[c] = b * (vx[c] - alpha * u[c]);
#pragma unroll
  for (int i = 0; i < RPT; ++i)
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      m[i][c] = fmaf(kx[i], d[c], alpha * m[i][c]);
      p[c] = fmaf(qx[i], m[i][c], p[c]);
    }
#pragma unroll
  for (int i = 0; i < RPT; ++i)
    __builtin_nontemporal_store(m[i], reinterpret_cast<f32x4*>(state_out + sbase + static_cast<int64_t>(rp * RPT + i) * DV));
  const f32x4 ot = decode_reduce<CQ>(p, red_o, lane, wave, cq);
  if (rp == 0) {
#pragma unroll
    for (int c = 0; c < 4; ++c) store_elt(o, nh * DV + col + c, scale * ot[c]);
  }
}

}  // namespace gdn
