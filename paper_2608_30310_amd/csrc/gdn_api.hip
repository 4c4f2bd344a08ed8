// GDN tail replay and chunked forward for MI355X (gfx950): kernels and the C ABI.
//
// Math (paper Section 2, Eq. 1, in the transposed layout M = S^T, d_k x d_v):
//   M_t = alpha_t M_{t-1} + k_t (beta_t (v_t - alpha_t M_{t-1}^T k_t))^T.
// The kernels evaluate it chunk by chunk (64 tokens) in the exact UT/WY
// rewrite: with G the in-chunk inclusive cumulative log-gate,
//   A  = strict_tril(diag(beta) K K^T * exp(G_i - G_j)),  T = (I + A)^-1,
//   R  = diag(beta) V - diag(beta e^G) K M0,               Delta = T R,
//   O  = scale (diag(e^G) Q M0 + (Q K^T * L) Delta),        L_ij = e^{G_i-G_j}, j <= i,
//   M1 = e^{G_last} M0 + K^T diag(e^{G_last - G}) Delta.
// Tail replay (Section 3, Eq. 2) is the same scan from M0 = 0 without outputs.
//
// Three launches per call, all on the caller's stream:
//   chunk_table  cu_seqlens -> first chunk of each sequence, (token, length) of each chunk
//   intra        per (chunk, value head), fully parallel: G, T and, for outputs, P = scale (Q K^T * L)
//   scan         per (sequence, value head, 32-column slice of d_v), sequential over the
//                sequence's chunks; the state slice stays in LDS for the whole sequence.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <limits>
#include <string>

#include "gdn_plan.h"
#include "gdn_tail_replay.h"

namespace gdn {
namespace {

thread_local std::string t_last_error;

constexpr int kThreads = 256;
constexpr int kBV = 32;   // d_v columns per scan workgroup

// ------------------------------------------------------------ element access
__device__ __forceinline__ float load_f32(const float* p, int64_t i) { return p[i]; }
__device__ __forceinline__ float load_f32(const uint16_t* p, int64_t i) {
  return __uint_as_float(static_cast<uint32_t>(p[i]) << 16);
}
__device__ __forceinline__ void store_from_f32(float* p, int64_t i, float x) { p[i] = x; }
__device__ __forceinline__ void store_from_f32(uint16_t* p, int64_t i, float x) {
  // float -> bfloat16, round to nearest, ties to even (finite values)
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  p[i] = static_cast<uint16_t>(u >> 16);
}

// ------------------------------------------------------------ chunk table
// One workgroup.  Sequence n owns chunks [seq_chunk[n], seq_chunk[n+1]); chunk
// c covers tokens [info.x, info.x + info.y) of the packed input.
__global__ __launch_bounds__(kThreads) void k_chunk_table(const int32_t* __restrict__ cu,
                                                          int32_t num_seqs,
                                                          int32_t* __restrict__ seq_chunk,
                                                          int2* __restrict__ chunk_info) {
  __shared__ int32_t scan[kThreads];
  __shared__ int32_t carry;
  const int tid = threadIdx.x;
  if (tid == 0) carry = 0;
  __syncthreads();
  for (int32_t base = 0; base < num_seqs; base += kThreads) {
    const int32_t n = base + tid;
    int32_t start = 0, len = 0, cnt = 0;
    if (n < num_seqs) {
      start = cu[n];
      len = cu[n + 1] - start;
      cnt = (len + kChunk - 1) / kChunk;
    }
    scan[tid] = cnt;
    __syncthreads();
    for (int off = 1; off < kThreads; off <<= 1) {
      const int32_t x = tid >= off ? scan[tid - off] : 0;
      __syncthreads();
      scan[tid] += x;
      __syncthreads();
    }
    const int32_t first = carry + scan[tid] - cnt;
    if (n < num_seqs) {
      seq_chunk[n] = first;
      for (int32_t j = 0; j < cnt; ++j)
        chunk_info[first + j] = make_int2(start + kChunk * j, min(kChunk, len - kChunk * j));
    }
    __syncthreads();
    if (tid == kThreads - 1) carry += scan[kThreads - 1];
    __syncthreads();
  }
  if (tid == 0) seq_chunk[num_seqs] = carry;
}

// ------------------------------------------------------------ intra-chunk
// grid = (num_chunks, Hv).  Writes, for chunk c and value head h:
//   G[c,h,i]   = sum_{j<=i} g_j                     (pad rows: g = 0)
//   T[c,h]     = (I + A)^-1, A_ij = beta_i e^{G_i-G_j} (k_i . k_j) for j < i
//   P[c,h]     = scale e^{G_i-G_j} (q_i . k_j) for j <= i, else 0   (outputs only)
template <typename TIn, int DK, bool FWD>
__global__ __launch_bounds__(kThreads) void k_intra(const int2* __restrict__ chunk_info,
                                                    int32_t hk, int32_t hv,
                                                    const TIn* __restrict__ q,
                                                    const TIn* __restrict__ k,
                                                    const float* __restrict__ g,
                                                    const float* __restrict__ beta,
                                                    float scale,
                                                    float* __restrict__ Tout,
                                                    float* __restrict__ Gout,
                                                    float* __restrict__ Pout) {
  __shared__ float Ks[kChunk][DK + 1];
  __shared__ float Qs[FWD ? kChunk : 1][DK + 1];
  __shared__ float As[kChunk][kChunk + 1];
  __shared__ float Ts[kChunk][kChunk + 1];
  __shared__ float Gs[kChunk], Bs[kChunk];

  const int tid = threadIdx.x;
  const int64_t c = blockIdx.x;
  const int h = blockIdx.y;
  const int kh = h / (hv / hk);
  const int2 info = chunk_info[c];
  const int start = info.x, len = info.y;

  for (int e = tid; e < kChunk * DK; e += kThreads) {
    const int i = e / DK, d = e % DK;
    const int64_t gi = (static_cast<int64_t>(start + i) * hk + kh) * DK + d;
    Ks[i][d] = i < len ? load_f32(k, gi) : 0.f;
    if (FWD) Qs[i][d] = i < len ? load_f32(q, gi) : 0.f;
  }
  if (tid < kChunk) {
    const int64_t gi = static_cast<int64_t>(start + tid) * hv + h;
    Gs[tid] = tid < len ? g[gi] : 0.f;
    Bs[tid] = tid < len ? beta[gi] : 0.f;
  }
  __syncthreads();
  if (tid == 0) {
    float run = 0.f;
    for (int i = 0; i < kChunk; ++i) { run += Gs[i]; Gs[i] = run; }
  }
  __syncthreads();

  for (int e = tid; e < kChunk * kChunk; e += kThreads) {
    const int i = e / kChunk, j = e % kChunk;
    float a = 0.f;
    if (j < i) {
      float dot = 0.f;
      for (int d = 0; d < DK; ++d) dot += Ks[i][d] * Ks[j][d];
      a = Bs[i] * __expf(Gs[i] - Gs[j]) * dot;
    }
    As[i][j] = a;
  }
  __syncthreads();

  // Unit lower-triangular inverse by forward substitution, one column per thread.
  if (tid < kChunk) {
    const int j = tid;
    for (int i = 0; i < kChunk; ++i) Ts[i][j] = (i == j) ? 1.f : 0.f;
    for (int i = j + 1; i < kChunk; ++i) {
      float s = 0.f;
      for (int l = j; l < i; ++l) s += As[i][l] * Ts[l][j];
      Ts[i][j] = -s;
    }
  }
  __syncthreads();

  const int64_t base = (c * hv + h);
  float* Tdst = Tout + base * kChunk * kChunk;
  for (int e = tid; e < kChunk * kChunk; e += kThreads) Tdst[e] = Ts[e / kChunk][e % kChunk];
  if (tid < kChunk) Gout[base * kChunk + tid] = Gs[tid];

  if (FWD) {
    float* Pdst = Pout + base * kChunk * kChunk;
    for (int e = tid; e < kChunk * kChunk; e += kThreads) {
      const int i = e / kChunk, j = e % kChunk;
      float p = 0.f;
      if (j <= i) {
        float dot = 0.f;
        for (int d = 0; d < DK; ++d) dot += Qs[i][d] * Ks[j][d];
        p = scale * __expf(Gs[i] - Gs[j]) * dot;
      }
      Pdst[e] = p;
    }
  }
}

// ------------------------------------------------------------ chunk scan
// grid = N * Hv * (d_v / 32), one workgroup per (sequence, value head, slice).
template <typename TIn, int DK, bool FWD>
__global__ __launch_bounds__(kThreads) void k_scan(const int32_t* __restrict__ cu,
                                                   const int32_t* __restrict__ seq_chunk,
                                                   int32_t hk, int32_t hv, int32_t dv,
                                                   const TIn* __restrict__ q,
                                                   const TIn* __restrict__ k,
                                                   const TIn* __restrict__ v,
                                                   const float* __restrict__ beta,
                                                   const float* __restrict__ Tin,
                                                   const float* __restrict__ Gin,
                                                   const float* __restrict__ Pin,
                                                   const float* __restrict__ state_in,
                                                   float scale,
                                                   TIn* __restrict__ o,
                                                   float* __restrict__ state_out) {
  constexpr int kRows = kChunk / (kThreads / kBV);   // 8 chunk rows per thread
  constexpr int kDRows = DK / (kThreads / kBV);      // state rows per thread
  __shared__ float Ks[kChunk][DK + 1];
  __shared__ float Qs[FWD ? kChunk : 1][DK + 1];
  __shared__ float Ms[DK][kBV];
  __shared__ float Rs[kChunk][kBV + 1];
  __shared__ float Ds[kChunk][kBV + 1];
  __shared__ float Ts[kChunk][kChunk + 1];
  __shared__ float Ps[FWD ? kChunk : 1][kChunk + 1];
  __shared__ float Gs[kChunk], Bs[kChunk], Ws[kChunk];

  const int tid = threadIdx.x;
  const int nslices = dv / kBV;
  const int unit = blockIdx.x;
  const int slice = unit % nslices;
  const int h = (unit / nslices) % hv;
  const int n = unit / (nslices * hv);
  const int kh = h / (hv / hk);
  const int col0 = slice * kBV;
  const int tok0 = cu[n];
  const int len = cu[n + 1] - tok0;
  const int chunk0 = seq_chunk[n];
  const int nch = (len + kChunk - 1) / kChunk;

  const int c = tid % kBV;        // column within the slice
  const int rg = tid / kBV;       // row group 0..7

  const int64_t sbase = (static_cast<int64_t>(n) * hv + h) * DK * dv + col0;
  for (int r = 0; r < kDRows; ++r) {
    const int d = rg + r * (kThreads / kBV);
    Ms[d][c] = state_in ? state_in[sbase + static_cast<int64_t>(d) * dv + c] : 0.f;
  }

  for (int ci = 0; ci < nch; ++ci) {
    const int t0 = tok0 + ci * kChunk;
    const int clen = min(kChunk, len - ci * kChunk);
    const int64_t cbase = static_cast<int64_t>(chunk0 + ci) * hv + h;
    // ---- stage the chunk
    for (int e = tid; e < kChunk * DK; e += kThreads) {
      const int i = e / DK, d = e % DK;
      const int64_t gi = (static_cast<int64_t>(t0 + i) * hk + kh) * DK + d;
      Ks[i][d] = i < clen ? load_f32(k, gi) : 0.f;
      if (FWD) Qs[i][d] = i < clen ? load_f32(q, gi) : 0.f;
    }
    for (int e = tid; e < kChunk * kChunk; e += kThreads) {
      Ts[e / kChunk][e % kChunk] = Tin[cbase * kChunk * kChunk + e];
      if (FWD) Ps[e / kChunk][e % kChunk] = Pin[cbase * kChunk * kChunk + e];
    }
    if (tid < kChunk) {
      Gs[tid] = Gin[cbase * kChunk + tid];
      Bs[tid] = tid < clen ? beta[static_cast<int64_t>(t0 + tid) * hv + h] : 0.f;
    }
    float vr[kRows];
    for (int r = 0; r < kRows; ++r) {
      const int i = rg + r * (kThreads / kBV);
      vr[r] = i < clen ? load_f32(v, (static_cast<int64_t>(t0 + i) * hv + h) * dv + col0 + c) : 0.f;
    }
    __syncthreads();

    // ---- K M0 (and Q M0), then R = diag(beta) V - diag(beta e^G) K M0
    const float glast = Gs[kChunk - 1];
    if (tid < kChunk) Ws[tid] = __expf(glast - Gs[tid]);
    float km[kRows], qm[kRows];
    for (int r = 0; r < kRows; ++r) { km[r] = 0.f; qm[r] = 0.f; }
    for (int d = 0; d < DK; ++d) {
      const float m = Ms[d][c];
      for (int r = 0; r < kRows; ++r) {
        const int i = rg + r * (kThreads / kBV);
        km[r] += Ks[i][d] * m;
        if (FWD) qm[r] += Qs[i][d] * m;
      }
    }
    for (int r = 0; r < kRows; ++r) {
      const int i = rg + r * (kThreads / kBV);
      Rs[i][c] = Bs[i] * (vr[r] - __expf(Gs[i]) * km[r]);
    }
    __syncthreads();

    // ---- Delta = T R
    for (int r = 0; r < kRows; ++r) {
      const int i = rg + r * (kThreads / kBV);
      float s = 0.f;
      for (int l = 0; l <= i; ++l) s += Ts[i][l] * Rs[l][c];
      Ds[i][c] = s;
    }
    __syncthreads();

    // ---- outputs O = scale e^G (Q M0) + P Delta
    if (FWD) {
      for (int r = 0; r < kRows; ++r) {
        const int i = rg + r * (kThreads / kBV);
        if (i < clen) {
          float s = scale * __expf(Gs[i]) * qm[r];
          for (int j = 0; j <= i; ++j) s += Ps[i][j] * Ds[j][c];
          store_from_f32(o, (static_cast<int64_t>(t0 + i) * hv + h) * dv + col0 + c, s);
        }
      }
    }
    // ---- state: M1 = e^{G_last} M0 + K^T diag(e^{G_last - G}) Delta
    const float eg = __expf(glast);
    for (int r = 0; r < kDRows; ++r) {
      const int d = rg + r * (kThreads / kBV);
      float s = 0.f;
      for (int i = 0; i < kChunk; ++i) s += Ks[i][d] * Ws[i] * Ds[i][c];
      Ms[d][c] = eg * Ms[d][c] + s;
    }
    __syncthreads();
  }

  if (state_out) {
    for (int r = 0; r < kDRows; ++r) {
      const int d = rg + r * (kThreads / kBV);
      state_out[sbase + static_cast<int64_t>(d) * dv + c] = Ms[d][c];
    }
  }
}

// ------------------------------------------------------------ host side
gdn_status fail(gdn_status st, const std::string& msg) {
  t_last_error = msg;
  return st;
}

gdn_status check_launch(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(GDN_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return GDN_OK;
}

struct Args {
  const gdn_shape* s;
  const Plan* p;
  const int32_t* cu;
  const void* q;
  const void* k;
  const void* v;
  const float* g;
  const float* beta;
  const float* state_in;
  void* o;
  float* state_out;
  char* ws;
  hipStream_t stream;
  void* const* events;   // NULL, or kNumStages + 1 hipEvent_t to record between stages
};

constexpr int32_t kNumStages = 3;
const char* const kStageNames[kNumStages] = {"chunk_table", "intra", "scan"};

gdn_status mark(const Args& a, int stage) {
  if (!a.events) return GDN_OK;
  const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(a.events[stage]), a.stream);
  if (e != hipSuccess)
    return fail(GDN_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
  return GDN_OK;
}

gdn_status mark_all(const Args& a) {
  for (int i = 0; i <= kNumStages; ++i) {
    const gdn_status st = mark(a, i);
    if (st != GDN_OK) return st;
  }
  return GDN_OK;
}

template <typename TIn, int DK, bool FWD>
gdn_status run(const Args& a) {
  const gdn_shape& s = *a.s;
  const Plan& p = *a.p;
  int32_t* seq_chunk = reinterpret_cast<int32_t*>(a.ws + p.off_seq_chunk);
  int2* chunk_info = reinterpret_cast<int2*>(a.ws + p.off_chunk_info);
  float* Tw = reinterpret_cast<float*>(a.ws + p.off_T);
  float* Gw = reinterpret_cast<float*>(a.ws + p.off_G);
  float* Pw = FWD ? reinterpret_cast<float*>(a.ws + p.off_P) : nullptr;

  gdn_status st = mark(a, 0);
  if (st != GDN_OK) return st;
  hipLaunchKernelGGL(k_chunk_table, dim3(1), dim3(kThreads), 0, a.stream, a.cu, s.num_seqs,
                     seq_chunk, chunk_info);
  st = check_launch("chunk_table launch");
  if (st != GDN_OK) return st;
  if ((st = mark(a, 1)) != GDN_OK) return st;
  if (p.num_chunks > 0) {
    hipLaunchKernelGGL((k_intra<TIn, DK, FWD>),
                       dim3(static_cast<uint32_t>(p.num_chunks), s.num_v_heads), dim3(kThreads), 0,
                       a.stream, chunk_info, s.num_k_heads, s.num_v_heads,
                       static_cast<const TIn*>(a.q), static_cast<const TIn*>(a.k), a.g, a.beta,
                       s.scale, Tw, Gw, Pw);
    st = check_launch("intra launch");
    if (st != GDN_OK) return st;
  }
  if ((st = mark(a, 2)) != GDN_OK) return st;
  const uint32_t units = static_cast<uint32_t>(s.num_seqs) * s.num_v_heads * (s.d_v / kBV);
  hipLaunchKernelGGL((k_scan<TIn, DK, FWD>), dim3(units), dim3(kThreads), 0, a.stream, a.cu,
                     seq_chunk, s.num_k_heads, s.num_v_heads, s.d_v,
                     static_cast<const TIn*>(a.q), static_cast<const TIn*>(a.k),
                     static_cast<const TIn*>(a.v), a.beta, Tw, Gw, Pw, a.state_in, s.scale,
                     static_cast<TIn*>(a.o), a.state_out);
  if ((st = check_launch("scan launch")) != GDN_OK) return st;
  return mark(a, 3);
}

template <bool FWD>
gdn_status dispatch(const Args& a) {
  const bool bf16 = a.s->qkv_dtype == GDN_BF16;
  if (a.s->d_k == 64)
    return bf16 ? run<uint16_t, 64, FWD>(a) : run<float, 64, FWD>(a);
  return bf16 ? run<uint16_t, 128, FWD>(a) : run<float, 128, FWD>(a);
}

gdn_status common_checks(const gdn_shape* shape, const int32_t* cu_host, const int32_t* cu,
                         bool fwd, Plan* plan, void* ws, size_t ws_bytes) {
  std::string err;
  const gdn_status st = make_plan(shape, cu_host, fwd, plan, &err);
  if (st != GDN_OK) return fail(st, err);
  if (shape->num_seqs > 0 && !cu) return fail(GDN_ERR_NULL_ARG, "cu_seqlens (device) is NULL");
  if (plan->bytes > 0 && !ws) return fail(GDN_ERR_WORKSPACE, "workspace is NULL");
  if (ws_bytes < plan->bytes)
    return fail(GDN_ERR_WORKSPACE, "workspace too small: need " + std::to_string(plan->bytes) +
                                       " bytes, got " + std::to_string(ws_bytes));
  if (reinterpret_cast<uintptr_t>(ws) % kAlign != 0)
    return fail(GDN_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  return GDN_OK;
}

}  // namespace
}  // namespace gdn

extern "C" {

gdn_status gdn_workspace_size(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                              int32_t with_outputs, size_t* bytes) {
  if (!bytes) return gdn::fail(GDN_ERR_NULL_ARG, "bytes is NULL");
  gdn::Plan plan;
  std::string err;
  const gdn_status st = gdn::make_plan(shape, cu_seqlens_host, with_outputs != 0, &plan, &err);
  if (st != GDN_OK) return gdn::fail(st, err);
  *bytes = plan.bytes;
  return GDN_OK;
}

}  // extern "C"

namespace gdn {
namespace {

gdn_status check_events(void* const* events, int32_t num_events) {
  if (!events) return fail(GDN_ERR_NULL_ARG, "stage_events is NULL");
  if (num_events != kNumStages + 1)
    return fail(GDN_ERR_BAD_SHAPE, "num_events must be gdn_num_stages() + 1");
  for (int i = 0; i < num_events; ++i)
    if (!events[i]) return fail(GDN_ERR_NULL_ARG, "a stage event is NULL");
  return GDN_OK;
}

gdn_status tail_replay_impl(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                            const int32_t* cu_seqlens, const void* k, const void* v,
                            const float* g, const float* beta, float* state_out,
                            void* workspace, size_t workspace_bytes, void* stream,
                            void* const* events) {
  gdn::Plan plan;
  gdn_status st = gdn::common_checks(shape, cu_seqlens_host, cu_seqlens, false, &plan,
                                     workspace, workspace_bytes);
  if (st != GDN_OK) return st;
  if (shape->num_seqs > 0 && !state_out) return gdn::fail(GDN_ERR_NULL_ARG, "state_out is NULL");
  if (plan.total_tokens > 0 && (!k || !v || !g || !beta))
    return gdn::fail(GDN_ERR_NULL_ARG, "k, v, g and beta must be non-NULL");
  const gdn::Args a{shape, &plan, cu_seqlens, nullptr, k, v, g, beta, nullptr,
                    nullptr, state_out, static_cast<char*>(workspace),
                    static_cast<hipStream_t>(stream), events};
  if (shape->num_seqs == 0) return mark_all(a);
  return gdn::dispatch<false>(a);
}

gdn_status chunk_forward_impl(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                              const int32_t* cu_seqlens, const void* q, const void* k,
                              const void* v, const float* g, const float* beta,
                              const float* state_in, void* o, float* state_out,
                              void* workspace, size_t workspace_bytes, void* stream,
                              void* const* events) {
  gdn::Plan plan;
  gdn_status st = gdn::common_checks(shape, cu_seqlens_host, cu_seqlens, true, &plan,
                                     workspace, workspace_bytes);
  if (st != GDN_OK) return st;
  if (plan.total_tokens > 0 && (!q || !k || !v || !g || !beta || !o))
    return gdn::fail(GDN_ERR_NULL_ARG, "q, k, v, g, beta and o must be non-NULL");
  if (state_in && state_out && state_in != state_out) {
    const size_t n = static_cast<size_t>(shape->num_seqs) * shape->num_v_heads * shape->d_k *
                     shape->d_v;
    const float* a0 = state_in;
    const float* a1 = state_in + n;
    const float* b0 = state_out;
    const float* b1 = state_out + n;
    if (a0 < b1 && b0 < a1)
      return gdn::fail(GDN_ERR_BAD_SHAPE, "state_out overlaps state_in without being equal");
  }
  const gdn::Args a{shape, &plan, cu_seqlens, q, k, v, g, beta, state_in,
                    o, state_out, static_cast<char*>(workspace),
                    static_cast<hipStream_t>(stream), events};
  if (shape->num_seqs == 0) return mark_all(a);
  return gdn::dispatch<true>(a);
}

}  // namespace
}  // namespace gdn

extern "C" {

gdn_status gdn_tail_replay(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                           const int32_t* cu_seqlens, const void* k, const void* v,
                           const float* g, const float* beta, float* state_out,
                           void* workspace, size_t workspace_bytes, void* stream) {
  return gdn::tail_replay_impl(shape, cu_seqlens_host, cu_seqlens, k, v, g, beta, state_out,
                               workspace, workspace_bytes, stream, nullptr);
}

gdn_status gdn_tail_replay_profiled(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                                    const int32_t* cu_seqlens, const void* k, const void* v,
                                    const float* g, const float* beta, float* state_out,
                                    void* workspace, size_t workspace_bytes, void* stream,
                                    void* const* stage_events, int32_t num_events) {
  const gdn_status st = gdn::check_events(stage_events, num_events);
  if (st != GDN_OK) return st;
  return gdn::tail_replay_impl(shape, cu_seqlens_host, cu_seqlens, k, v, g, beta, state_out,
                               workspace, workspace_bytes, stream, stage_events);
}

gdn_status gdn_chunk_forward(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                             const int32_t* cu_seqlens, const void* q, const void* k,
                             const void* v, const float* g, const float* beta,
                             const float* state_in, void* o, float* state_out,
                             void* workspace, size_t workspace_bytes, void* stream) {
  return gdn::chunk_forward_impl(shape, cu_seqlens_host, cu_seqlens, q, k, v, g, beta,
                                 state_in, o, state_out, workspace, workspace_bytes, stream,
                                 nullptr);
}

gdn_status gdn_chunk_forward_profiled(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                                      const int32_t* cu_seqlens, const void* q, const void* k,
                                      const void* v, const float* g, const float* beta,
                                      const float* state_in, void* o, float* state_out,
                                      void* workspace, size_t workspace_bytes, void* stream,
                                      void* const* stage_events, int32_t num_events) {
  const gdn_status st = gdn::check_events(stage_events, num_events);
  if (st != GDN_OK) return st;
  return gdn::chunk_forward_impl(shape, cu_seqlens_host, cu_seqlens, q, k, v, g, beta,
                                 state_in, o, state_out, workspace, workspace_bytes, stream,
                                 stage_events);
}

int32_t gdn_num_stages(int32_t with_outputs) {
  (void)with_outputs;
  return gdn::kNumStages;
}

const char* gdn_stage_name(int32_t with_outputs, int32_t stage) {
  (void)with_outputs;
  if (stage < 0 || stage >= gdn::kNumStages) return "";
  return gdn::kStageNames[stage];
}

int64_t gdn_replay_len(int64_t m, int64_t ratio_num, int64_t ratio_den) {
  if (m < 0 || ratio_num < 0 || ratio_den <= 0) return -1;
  if (ratio_num != 0 && m > std::numeric_limits<int64_t>::max() / ratio_num) return -1;
  const int64_t num = m * ratio_num;
  return num / ratio_den + (num % ratio_den != 0 ? 1 : 0);
}

const char* gdn_status_string(gdn_status status) {
  switch (status) {
    case GDN_OK: return "GDN_OK: success";
    case GDN_ERR_NULL_ARG: return "GDN_ERR_NULL_ARG: a required pointer is NULL";
    case GDN_ERR_BAD_SHAPE: return "GDN_ERR_BAD_SHAPE: inconsistent shape or aliasing";
    case GDN_ERR_BAD_SEQLENS: return "GDN_ERR_BAD_SEQLENS: cu_seqlens must start at 0 and be non-decreasing";
    case GDN_ERR_UNSUPPORTED: return "GDN_ERR_UNSUPPORTED: configuration not supported";
    case GDN_ERR_WORKSPACE: return "GDN_ERR_WORKSPACE: workspace missing, misaligned or too small";
    case GDN_ERR_HIP: return "GDN_ERR_HIP: HIP runtime error";
  }
  return "unknown gdn_status";
}

const char* gdn_last_error(void) { return gdn::t_last_error.c_str(); }

}  // extern "C"
