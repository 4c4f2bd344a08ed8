// Kernels of the linear-attention layer block around the recurrence (paper
// Section 3: the replayed hiddens pass through the layer's projections before
// Eq. 2).  Two memory-bound passes, fp32 arithmetic:
//
//   k_la_prep     the short causal depthwise convolution (4 taps, zero history
//                 before each sequence's first token) over the q, k, v columns
//                 of the in-projection, SiLU, the L2 norm of every q and k head,
//                 and the gates g = -exp(A_log) softplus(a + dt_bias),
//                 beta = sigmoid(b);
//   k_gated_norm  y = o / sqrt(mean(o^2) + eps) * w_norm * silu(z) per
//                 (token, value head), written as bf16 for the out-projection.
//
// Both give each thread eight consecutive channels (one 16-byte bf16 access,
// two for fp32), so a head of d channels is d / 8 adjacent lanes and its norm
// is a lane-exchange reduction inside the wave.
#pragma once

#include "gdn_decode.h"

namespace gdn {

constexpr int kPrepThreads = 256;
constexpr int kPrepChans = 256;   // channels per prep workgroup (32 threads x 8)
// tokens per prep workgroup when each thread takes TPT consecutive tokens
constexpr int prep_tokens(int tpt) { return kPrepThreads / (kPrepChans / 8) * tpt; }
constexpr int kConvTaps = 4;
constexpr int kNormThreads = 256;

template <typename T>
__device__ __forceinline__ void store8(T* __restrict__ p, const float (&x)[8]) {
  if constexpr (sizeof(T) == 2) {
    // the hardware pair conversion rounds to nearest even, as f2bf does
    u32x4 w;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const f32x2 pair = {x[2 * j], x[2 * j + 1]};
      w[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(pair, bf16x2));
    }
    *reinterpret_cast<u32x4*>(p) = w;
  } else {
    reinterpret_cast<f32x4*>(p)[0] = f32x4{x[0], x[1], x[2], x[3]};
    reinterpret_cast<f32x4*>(p)[1] = f32x4{x[4], x[5], x[6], x[7]};
  }
}

// x sigmoid(x) with the hardware exponential and reciprocal (about 1e-7
// relative; x far below zero gives exp = inf, rcp = 0 and -0)
__device__ __forceinline__ float silu_f(float x) { return x * __builtin_amdgcn_rcpf(1.0f + __expf(-x)); }

// Sequence of token t (0 <= t < cu[n_seqs]): the largest n with cu[n] <= t,
// which skips empty sequences.
__device__ __forceinline__ int seq_of(const int32_t* __restrict__ cu, int n_seqs, int t) {
  int lo = 0, hi = n_seqs - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) / 2;
    if (cu[mid] <= t) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// One unit of k_la_prep: channel slab `slab` (or the gates when slab ==
// chan_slabs) of token block `tb`.
template <typename TP, typename TQ, int DK, int DV, int TPT>
__device__ __forceinline__ void prep_unit(int slab, int tb, int32_t T, int32_t n_seqs,
                                          const int32_t* __restrict__ cu, int32_t hk, int32_t hv,
                                          const TP* __restrict__ P, int64_t ldp, int32_t chan0,
                                          int32_t chan_slabs, const float* __restrict__ conv_w,
                                          const float* __restrict__ a_log, const float* __restrict__ dt_bias,
                                          float l2_eps, TQ* __restrict__ q, TQ* __restrict__ k,
                                          TQ* __restrict__ v, float* __restrict__ g, float* __restrict__ beta,
                                          float (*wlds)[kPrepChans]) {
  constexpr int H = kConvTaps - 1;
  const int cq = hk * DK, cv = hv * DV, nch = 2 * cq + cv;
  const int t0 = tb * prep_tokens(TPT);
  const int tid = threadIdx.x;

  if (slab == chan_slabs) {   // gates
    const int ca = nch - chan0;
    const int t1 = min(T, t0 + prep_tokens(TPT));
    for (int i = tid; i < (t1 - t0) * hv; i += kPrepThreads) {
      const int t = t0 + i / hv, h = i % hv;
      const TP* row = P + static_cast<int64_t>(t) * ldp;
      const float a = load_elt(row, ca + h) + dt_bias[h];
      const float b = load_elt(row, ca + hv + h);
      const float sp = a > 20.0f ? a : log1pf(expf(a));
      g[static_cast<int64_t>(t) * hv + h] = -expf(a_log[h]) * sp;
      beta[static_cast<int64_t>(t) * hv + h] = 1.0f / (1.0f + expf(-b));
    }
    return;
  }

  const int tt = t0 + TPT * (tid / (kPrepChans / 8));   // this thread's first token
  const int cg = tid % (kPrepChans / 8);
  const int c0 = chan0 + (slab * (kPrepChans / 8) + cg) * 8;
  const bool any = c0 < nch && tt < T;   // idle lanes still join the lane exchanges
  // Every global load of the unit is issued before anything waits: the
  // slab's conv taps (one coalesced 16-byte load per thread, channel
  // slab * 256 + tid) and the rows tt - 3 .. tt + TPT - 1 of this thread's
  // eight channels, each loaded once for the TPT tokens that use it (rows
  // before a token's sequence are zeroed afterwards).
  const int ch = chan0 + slab * kPrepChans + tid;
  const float4 w4 = ch < nch ? reinterpret_cast<const float4*>(conv_w)[ch] : make_float4(0.f, 0.f, 0.f, 0.f);
  float u[TPT + H][8];
  int first[TPT];
  if (any) {
    const TP* col = P + (c0 - chan0);
#pragma unroll
    for (int r = 0; r < TPT + H; ++r) {
      const int tr = tt - H + r;
      if (tr >= 0 && tr < T) {
        load_run<TP, 8>(col + static_cast<int64_t>(tr) * ldp, u[r]);
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) u[r][e] = 0.0f;
      }
    }
    // first token of each token's sequence (empty sequences skipped)
    int sq = seq_of(cu, n_seqs, tt);
#pragma unroll
    for (int i = 0; i < TPT; ++i) {
      while (sq + 1 < n_seqs && cu[sq + 1] <= tt + i) ++sq;
      first[i] = cu[sq];
    }
  }
  // the taps, tap-major in LDS; each thread then reads its eight channels of
  // each tap as two 16-byte LDS reads
  lds_barrier();   // the previous unit's LDS readers are done
  wlds[0][tid] = w4.x;
  wlds[1][tid] = w4.y;
  wlds[2][tid] = w4.z;
  wlds[3][tid] = w4.w;
  lds_barrier();
  float w[kConvTaps][8];
#pragma unroll
  for (int j = 0; j < kConvTaps; ++j) {
    const f32x4 lo = *reinterpret_cast<const f32x4*>(&wlds[j][cg * 8]);
    const f32x4 hi = *reinterpret_cast<const f32x4*>(&wlds[j][cg * 8 + 4]);
#pragma unroll
    for (int e = 0; e < 4; ++e) { w[j][e] = lo[e]; w[j][4 + e] = hi[e]; }
  }
  const int sec = c0 < cq ? 0 : (c0 < 2 * cq ? 1 : 2);
#pragma unroll
  for (int i = 0; i < TPT; ++i) {
    const int t = tt + i;
    const bool active = any && t < T;
    float c[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) c[e] = 0.0f;
    if (active) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        float acc = 0.0f;
#pragma unroll
        for (int j = 0; j < kConvTaps; ++j)   // before the sequence: zero history
          acc += w[j][e] * (t - H + j >= first[i] ? u[i + j][e] : 0.0f);
        c[e] = silu_f(acc);
      }
    }
    float ss = 0.0f;
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += c[e] * c[e];
    // sum of squares over the head (DK / 8 lanes); used by q and k lanes only
#pragma unroll
    for (int off = 1; off < DK / 8; off <<= 1) ss += __shfl_xor(ss, off, kWave);
    if (!active) continue;
    if (sec < 2) {
      const float r = rsqrtf(ss + l2_eps);
#pragma unroll
      for (int e = 0; e < 8; ++e) c[e] *= r;
    }
    TQ* dst;
    if (sec == 0) dst = q + static_cast<int64_t>(t) * cq + c0;
    else if (sec == 1) dst = k + static_cast<int64_t>(t) * cq + (c0 - cq);
    else dst = v + static_cast<int64_t>(t) * cv + (c0 - 2 * cq);
    store8(dst, c);
  }
}

// P [T, ldp] (TP) holds the in-projection from channel chan0 on: q|k|v
// channels chan0 .. 2 cq + cv, then a [hv], then b [hv].  chan0 = 0 computes
// q, k and v; chan0 = cq (no queries) k and v only.
// One thread per (TPT consecutive tokens, eight channels): a workgroup covers
// prep_tokens(TPT) tokens x kPrepChans channels, thread (tok, cg) = (tid / 32,
// tid % 32), and loads each row its taps need once.  TPT = 4 when there are
// enough tokens to keep every workgroup of the grid busy (fewer loads per
// token, more of them in flight per thread), else 1 (more units, more waves).
// Units: chan_slabs channel slabs plus one gate slab per token block; unit u
// is xcd-remapped to logical index token_block * (chan_slabs + 1) + slab, so
// an XCD streams whole rows of P, token after token.  The
// grid is sized to the machine (a few workgroups per CU) and strides over the
// units, so waves live long enough to keep many loads in flight: one short
// wave per unit leaves the CUs mostly waiting for wave launches.  The stride
// is a multiple of 8, so a unit runs on the XCD its remap assumes.
template <typename TP, typename TQ, int DK, int DV, int TPT>
__global__ __launch_bounds__(kPrepThreads)
void k_la_prep(int32_t T, int32_t n_seqs, const int32_t* __restrict__ cu, int32_t hk, int32_t hv,
               const TP* __restrict__ P, int64_t ldp, int32_t chan0, int32_t chan_slabs,
               int32_t token_blocks, const float* __restrict__ conv_w, const float* __restrict__ a_log,
               const float* __restrict__ dt_bias, float l2_eps, TQ* __restrict__ q,
               TQ* __restrict__ k, TQ* __restrict__ v, float* __restrict__ g,
               float* __restrict__ beta) {
  __shared__ __attribute__((aligned(16))) float wlds[kConvTaps][kPrepChans];
  const int total = token_blocks * (chan_slabs + 1);
  for (int unit = blockIdx.x; unit < total; unit += gridDim.x) {   // uniform per workgroup
    const int logical = xcd_remap(unit, total);
    const int slabs = chan_slabs + 1;
    prep_unit<TP, TQ, DK, DV, TPT>(logical % slabs, logical / slabs, T, n_seqs, cu, hk, hv, P,
                              ldp, chan0, chan_slabs, conv_w, a_log, dt_bias, l2_eps, q, k, v, g, beta,
                              wlds);
  }
}


// One group of k_gated_norm: the eight channels from element e = 8 i of
// y [T, hv DV]; `active` false for the padding lanes past the end, which only
// join the lane exchange.
template <typename TO, typename TP, int DV>
__device__ __forceinline__ void norm_group(int64_t i, bool active, int32_t cv, const TO* __restrict__ o,
                                           const TP* __restrict__ P, int64_t ldp, int32_t col_z,
                                           const float* __restrict__ w_norm, float eps, uint16_t* __restrict__ y) {
  const int64_t e = i * 8;
  const int64_t t = e / cv;
  const int c = static_cast<int>(e - t * cv);
  float ov[8], zv[8];
  if (active) {
    load_run<TO, 8>(o + e, ov);
    load_run<TP, 8>(P + t * ldp + col_z + c, zv);
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) ov[j] = zv[j] = 0.0f;
  }
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < 8; ++j) ss += ov[j] * ov[j];
#pragma unroll
  for (int off = 1; off < DV / 8; off <<= 1) ss += __shfl_xor(ss, off, kWave);
  const float r = rsqrtf(ss * (1.0f / DV) + eps);
  if (!active) return;
  const int cj = c % DV;
  const f32x4 w0 = *reinterpret_cast<const f32x4*>(w_norm + cj);
  const f32x4 w1 = *reinterpret_cast<const f32x4*>(w_norm + cj + 4);
  float out[8];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    out[j] = ov[j] * r * w0[j] * silu_f(zv[j]);
    out[4 + j] = ov[4 + j] * r * w1[j] * silu_f(zv[4 + j]);
  }
  store8(y + e, out);
}

// o [T, hv, DV] (TO); z at P[t, col_z + h DV + j] (TP); y [T, hv DV] bf16.
// One thread per eight channels, groups = T hv DV / 8, a whole head (DV / 8
// lanes) active or idle together; the grid strides over the groups (sized to
// the machine, as for k_la_prep).
template <typename TO, typename TP, int DV>
__global__ __launch_bounds__(kNormThreads)
void k_gated_norm(int64_t groups, int32_t cv, const TO* __restrict__ o, const TP* __restrict__ P,
                  int64_t ldp, int32_t col_z, const float* __restrict__ w_norm, float eps,
                  uint16_t* __restrict__ y) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kNormThreads;
  for (int64_t base = static_cast<int64_t>(blockIdx.x) * kNormThreads; base < groups; base += stride) {
    const int64_t i = base + threadIdx.x;
    norm_group<TO, TP, DV>(i, i < groups, cv, o, P, ldp, col_z, w_norm, eps, y);
  }
}

}  // namespace gdn
