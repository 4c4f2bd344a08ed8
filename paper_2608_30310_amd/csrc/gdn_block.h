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
constexpr int kPrepTokens = 16;   // tokens per workgroup: the conv window slides in registers
constexpr int kConvTaps = 4;
constexpr int kNormThreads = 256;

template <typename T>
__device__ __forceinline__ void store8(T* __restrict__ p, const float (&x)[8]) {
  if constexpr (sizeof(T) == 2) {
    u32x4 w;
#pragma unroll
    for (int j = 0; j < 4; ++j) w[j] = f2bf(x[2 * j]) | (static_cast<uint32_t>(f2bf(x[2 * j + 1])) << 16);
    *reinterpret_cast<u32x4*>(p) = w;
  } else {
    reinterpret_cast<f32x4*>(p)[0] = f32x4{x[0], x[1], x[2], x[3]};
    reinterpret_cast<f32x4*>(p)[1] = f32x4{x[4], x[5], x[6], x[7]};
  }
}

__device__ __forceinline__ float silu_f(float x) { return x / (1.0f + expf(-x)); }

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

// P [T, ldp] (TP) holds the in-projection from channel chan0 on: q|k|v
// channels chan0 .. 2 cq + cv, then a [hv], then b [hv].  chan0 = 0 computes
// q, k and v; chan0 = cq (no queries) k and v only.  Grid: xcd-remapped
// 1-D, logical index = slab * token_blocks + token_block, slabs = chan_slabs
// channel slabs of 2048 channels plus one gate slab.
template <typename TP, typename TQ, int DK, int DV>
__global__ __launch_bounds__(kPrepThreads)
void k_la_prep(int32_t T, int32_t n_seqs, const int32_t* __restrict__ cu, int32_t hk, int32_t hv,
               const TP* __restrict__ P, int64_t ldp, int32_t chan0, int32_t chan_slabs,
               int32_t token_blocks, const float* __restrict__ conv_w, const float* __restrict__ a_log,
               const float* __restrict__ dt_bias, float l2_eps, TQ* __restrict__ q,
               TQ* __restrict__ k, TQ* __restrict__ v, float* __restrict__ g,
               float* __restrict__ beta) {
  const int total = token_blocks * (chan_slabs + 1);
  const int logical = xcd_remap(blockIdx.x, total);
  const int slab = logical / token_blocks, tb = logical % token_blocks;
  const int cq = hk * DK, cv = hv * DV, nch = 2 * cq + cv;
  const int t0 = tb * kPrepTokens;
  const int t1 = min(T, t0 + kPrepTokens);
  const int tid = threadIdx.x;

  if (slab == chan_slabs) {   // gates
    const int ca = nch - chan0;
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

  const int c0 = chan0 + (slab * kPrepThreads + tid) * 8;
  const bool active = c0 < nch;      // idle lanes still join the lane exchanges
  const int sec = c0 < cq ? 0 : (c0 < 2 * cq ? 1 : 2);
  TQ* dst;
  int64_t ld;
  if (sec == 0) { dst = q + c0; ld = cq; }
  else if (sec == 1) { dst = k + (c0 - cq); ld = cq; }
  else { dst = v + (c0 - 2 * cq); ld = cv; }
  float w[8][kConvTaps];
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    const float4 t4 = active ? reinterpret_cast<const float4*>(conv_w)[c0 + i] : make_float4(0.f, 0.f, 0.f, 0.f);
    w[i][0] = t4.x; w[i][1] = t4.y; w[i][2] = t4.z; w[i][3] = t4.w;
  }
  const TP* col = P + (c0 - chan0);

  int n = seq_of(cu, n_seqs, t0);
  int start = cu[n];
  int next = cu[n + 1];
  float u1[8], u2[8], u3[8];   // u[t-1], u[t-2], u[t-3]
  auto row = [&](int t, float (&x)[8]) {
    if (active && t >= start) {
      load_run<TP, 8>(col + static_cast<int64_t>(t) * ldp, x);
    } else {
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = 0.0f;
    }
  };
  row(t0 - 1, u1);
  row(t0 - 2, u2);
  row(t0 - 3, u3);
  for (int t = t0; t < t1; ++t) {
    if (t == next) {   // a sequence starts here: its convolution history is zero
      while (cu[n + 1] <= t) ++n;
      start = t;
      next = cu[n + 1];
#pragma unroll
      for (int i = 0; i < 8; ++i) u1[i] = u2[i] = u3[i] = 0.0f;
    }
    float u0[8];
    row(t, u0);
    float c[8], ss = 0.0f;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const float s = w[i][0] * u3[i] + w[i][1] * u2[i] + w[i][2] * u1[i] + w[i][3] * u0[i];
      c[i] = silu_f(s);
      ss += c[i] * c[i];
    }
    // sum of squares over the head (DK / 8 lanes); used by q and k lanes only
#pragma unroll
    for (int off = 1; off < DK / 8; off <<= 1) ss += __shfl_xor(ss, off, kWave);
    if (sec < 2) {
      const float r = rsqrtf(ss + l2_eps);
#pragma unroll
      for (int i = 0; i < 8; ++i) c[i] *= r;
    }
    if (active) store8(dst + static_cast<int64_t>(t) * ld, c);
#pragma unroll
    for (int i = 0; i < 8; ++i) { u3[i] = u2[i]; u2[i] = u1[i]; u1[i] = u0[i]; }
  }
}

// o [T, hv, DV] (TO); z at P[t, col_z + h DV + j] (TP); y [T, hv DV] bf16.
// One thread per eight channels, groups = T hv DV / 8.
template <typename TO, typename TP, int DV>
__global__ __launch_bounds__(kNormThreads)
void k_gated_norm(int64_t groups, int32_t cv, const TO* __restrict__ o, const TP* __restrict__ P,
                  int64_t ldp, int32_t col_z, const float* __restrict__ w_norm, float eps,
                  uint16_t* __restrict__ y) {
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kNormThreads + threadIdx.x;
  const bool active = i < groups;    // whole heads are active or idle together
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
  float out[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) out[j] = ov[j] * r * w_norm[cj + j] * silu_f(zv[j]);
  store8(y + e, out);
}

}  // namespace gdn
