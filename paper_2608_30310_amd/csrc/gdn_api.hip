// GDN tail replay and chunked forward for MI355X (gfx950): the C ABI.
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
// Two launches per call, both on the caller's stream:
//   intra  per (chunk slot, value head), fully parallel: T (and P) as split
//          bf16 MFMA fragments plus per-row scalars (gdn_intra.h)
//   scan   per (sequence, value head), sequential over the sequence's chunks
//          with the state in registers (gdn_scan.h)
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <limits>
#include <string>

#include "gdn_intra.h"
#include "gdn_plan.h"
#include "gdn_scan.h"
#include "gdn_tail_replay.h"

namespace gdn {
namespace {

thread_local std::string t_last_error;

constexpr int kThreads = 256;
// grid limits in make_plan assume <= 1024 work items per (sequence, head) in any grid dimension
static_assert(kThreads <= 256 && kColsThreads <= 256 && head_threads(128) <= 1024, "grid limits");

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

constexpr int32_t kNumStages = 2;
const char* const kStageNames[kNumStages] = {"intra", "scan"};

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

template <typename TIn, int DK, int DV, bool FWD>
gdn_status run(const Args& a) {
  const gdn_shape& s = *a.s;
  const Plan& p = *a.p;
  u32x4* Kw = reinterpret_cast<u32x4*>(a.ws + p.off_K);
  u32x4* Tw = reinterpret_cast<u32x4*>(a.ws + p.off_T);
  float* Sw = reinterpret_cast<float*>(a.ws + p.off_S);
  u32x4* Pw = FWD ? reinterpret_cast<u32x4*>(a.ws + p.off_P) : nullptr;

  gdn_status st = mark(a, 0);
  if (st != GDN_OK) return st;
  if (p.num_slots > 0) {
    hipLaunchKernelGGL((k_intra<TIn, DK, FWD>),
                       dim3(static_cast<uint32_t>(p.num_slots), s.num_v_heads), dim3(kThreads), 0,
                       a.stream, a.cu, s.num_seqs, s.num_k_heads, s.num_v_heads,
                       static_cast<const TIn*>(a.q), static_cast<const TIn*>(a.k), a.g, a.beta,
                       s.scale, Kw, Tw, Sw, Pw);
    if ((st = check_launch("intra launch")) != GDN_OK) return st;
  }
  if ((st = mark(a, 1)) != GDN_OK) return st;
  // The column-split kernel has the shortest chunk latency but one workgroup
  // per CU; use it when its grid fits on the chip at once, else the whole-head
  // kernel (4x the columns per CU, two waves per SIMD).
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return fail(GDN_ERR_HIP, "querying the device");
  const uint32_t heads = static_cast<uint32_t>(s.num_seqs) * s.num_v_heads;
  const uint32_t col_groups = heads * (s.d_v / kColsPerGroup);
  if (col_groups <= static_cast<uint32_t>(cus)) {
    hipLaunchKernelGGL((k_scan_cols<TIn, DK, FWD>), dim3(col_groups), dim3(kColsThreads), 0, a.stream,
                       a.cu, s.num_k_heads, s.num_v_heads, s.d_v, static_cast<const TIn*>(a.v), Kw, Tw, Sw,
                       Pw, a.state_in, static_cast<TIn*>(a.o), a.state_out);
  } else {
    hipLaunchKernelGGL((k_scan_head<TIn, DK, DV, FWD>), dim3(heads), dim3(head_threads(DV)), 0, a.stream,
                       a.cu, s.num_k_heads, s.num_v_heads, static_cast<const TIn*>(a.v), Kw, Tw, Sw, Pw,
                       a.state_in, static_cast<TIn*>(a.o), a.state_out);
  }
  if ((st = check_launch("scan launch")) != GDN_OK) return st;
  return mark(a, 2);
}

template <int DK, int DV, bool FWD>
gdn_status run_dtype(const Args& a) {
  return a.s->qkv_dtype == GDN_BF16 ? run<uint16_t, DK, DV, FWD>(a) : run<float, DK, DV, FWD>(a);
}

template <bool FWD>
gdn_status dispatch(const Args& a) {
  const int dk = a.s->d_k, dv = a.s->d_v;
  if (dk == 64) return dv == 64 ? run_dtype<64, 64, FWD>(a) : run_dtype<64, 128, FWD>(a);
  return dv == 64 ? run_dtype<128, 64, FWD>(a) : run_dtype<128, 128, FWD>(a);
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
  if (reinterpret_cast<uintptr_t>(k) % 16 != 0 || reinterpret_cast<uintptr_t>(v) % 16 != 0)
    return gdn::fail(GDN_ERR_UNSUPPORTED, "k and v must be 16-byte aligned");
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
  if (reinterpret_cast<uintptr_t>(q) % 16 != 0 || reinterpret_cast<uintptr_t>(k) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(v) % 16 != 0 || reinterpret_cast<uintptr_t>(o) % 16 != 0)
    return gdn::fail(GDN_ERR_UNSUPPORTED, "q, k, v and o must be 16-byte aligned");
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
