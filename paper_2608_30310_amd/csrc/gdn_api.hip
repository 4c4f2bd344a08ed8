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
#include <mutex>
#include <string>

#include "gdn_decode.h"
#include "gdn_intra.h"
#include "gdn_plan.h"
#include "gdn_scan.h"
#include "gdn_tail_replay.h"

namespace gdn {
namespace {

constexpr int kThreads = 256;
// grid limits in make_plan assume <= 1024 work items per (sequence, head) in any
// grid dimension; the column-split scan's grid is bounded by the CU count instead
static_assert(kThreads <= 256 && kDecodeThreads <= 1024 && head_threads(128) <= 1024, "grid limits");

// ------------------------------------------------------------ host side
gdn_status fail(gdn_status st, const std::string& msg) {
  set_last_error(msg);
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
  void* const* events;   // NULL, or num_stages(fwd) + 1 hipEvent_t to record between stages
};

// Stages of a call: tail replay {intra, scan, combine} (combine is empty
// unless the chain runs in two halves), forward {intra, scan}.
constexpr int32_t kMaxStages = 3;
constexpr int32_t num_stages(bool fwd) { return fwd ? 2 : 3; }
const char* const kStageNames[kMaxStages] = {"intra", "scan", "combine"};

gdn_status mark(const Args& a, int stage) {
  if (!a.events) return GDN_OK;
  const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(a.events[stage]), a.stream);
  if (e != hipSuccess)
    return fail(GDN_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
  return GDN_OK;
}

gdn_status mark_all(const Args& a, bool fwd) {
  for (int i = 0; i <= num_stages(fwd); ++i) {
    const gdn_status st = mark(a, i);
    if (st != GDN_OK) return st;
  }
  return GDN_OK;
}

template <typename TIn, int DK, bool FWD>
gdn_status launch_intra(const gdn_shape& s, const Plan& p, const int32_t* cu, const void* q, const void* k,
                        const float* g, const float* beta, char* ws, hipStream_t stream) {
  if (p.num_slots == 0) return GDN_OK;
  const dim3 block(kThreads);
  const auto launch = [&](auto kernel, uint32_t heads_per_group) {
    hipLaunchKernelGGL(kernel, dim3(static_cast<uint32_t>(p.num_slots), s.num_v_heads / heads_per_group), block, 0,
                       stream, cu, s.num_seqs, s.num_k_heads, s.num_v_heads, static_cast<const TIn*>(q),
                       static_cast<const TIn*>(k), g, beta, s.scale, reinterpret_cast<u32x4*>(ws + p.off_K),
                       reinterpret_cast<u32x4*>(ws + p.off_T), reinterpret_cast<float*>(ws + p.off_S),
                       FWD ? reinterpret_cast<u32x4*>(ws + p.off_P) : nullptr);
  };
  // tail replay: one workgroup per two value heads of a key head where the
  // group allows and one workgroup per head would take more than one round of
  // the chip (seven per CU): the key rows are loaded and K K^T formed once for
  // both heads, which saves work in a throughput batch, while a grid that fits
  // at once finishes sooner with a head per workgroup
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return fail(GDN_ERR_HIP, "querying the device");
  const bool pair = !FWD && (s.num_v_heads / s.num_k_heads) % 2 == 0 &&
                    p.num_slots * s.num_v_heads > 7 * static_cast<int64_t>(cus);
  if (pair) launch(k_intra<TIn, DK, FWD, FWD ? 1 : 2>, 2);
  else launch(k_intra<TIn, DK, FWD, 1>, 1);
  return check_launch("intra launch");
}

// The column-split scan has the shortest chunk latency but one workgroup per
// CU; it is used when its grid fits on the chip at once.  Tail replay of bf16
// inputs whose split grid (the two halves of the chain side by side and the
// second half's transition) also fits runs split, which halves the chain.
// When the 32-wide grid does not fit, tail replay of bf16 inputs takes the
// wide column scan (two tiles per wave, two workgroups per CU: throughput) and
// everything else the whole-head scan.
gdn_status cols_fit(const gdn_shape& s, bool* fits, uint32_t* col_groups, int* cus_out = nullptr) {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return fail(GDN_ERR_HIP, "querying the device");
  *col_groups = static_cast<uint32_t>(s.num_seqs) * s.num_v_heads * (s.d_v / kColsPerGroup);
  *fits = *col_groups <= static_cast<uint32_t>(cus);
  if (cus_out) *cus_out = cus;
  return GDN_OK;
}

// `marks` (tail replay only, may be NULL): the call whose stage events are
// recorded; its combine stage starts before k_state_combine.
template <typename TIn, int DK, int DV, bool FWD>
gdn_status launch_scan(const gdn_shape& s, const Plan& p, const int32_t* cu, const void* v, const void* k,
                       const void* q, const float* state_in, void* o, float* state_out, char* ws, hipStream_t stream,
                       const Args* marks = nullptr, bool* combined = nullptr) {
  const u32x4* Kw = reinterpret_cast<const u32x4*>(ws + p.off_K);
  const u32x4* Tw = reinterpret_cast<const u32x4*>(ws + p.off_T);
  const float* Sw = reinterpret_cast<const float*>(ws + p.off_S);
  const u32x4* Pw = FWD ? reinterpret_cast<const u32x4*>(ws + p.off_P) : nullptr;
  bool fits = false;
  uint32_t col_groups = 0;
  int cus = 0;
  gdn_status st = cols_fit(s, &fits, &col_groups, &cus);
  if (st != GDN_OK) return st;
  constexpr bool kWide = !FWD && sizeof(TIn) == 2;   // tail replay, bf16 inputs
  if constexpr (kWide) {
    if (p.split && split_groups(s) <= cus) {
      // two half-length chains side by side, then state = A state + M''
      float* m2 = reinterpret_cast<float*>(ws + p.off_M2);
      float* a2 = reinterpret_cast<float*>(ws + p.off_A2);
      hipLaunchKernelGGL((k_scan_cols_split<TIn, DK>), dim3(static_cast<uint32_t>(split_groups(s))),
                         dim3(cols_split_threads()), 0, stream,
                         static_cast<int32_t>(split_first_groups(s)), cu, s.num_k_heads, s.num_v_heads, s.d_v, static_cast<const TIn*>(v), static_cast<const TIn*>(k),
                         static_cast<const TIn*>(q), Kw, Tw, Sw, state_out, m2, a2);
      if ((st = check_launch("split scan launch")) != GDN_OK) return st;
      if (marks && (st = mark(*marks, 2)) != GDN_OK) return st;
      if (combined) *combined = true;
      hipLaunchKernelGGL((k_state_combine<DK>),
                         dim3(static_cast<uint32_t>(s.num_seqs) * s.num_v_heads * (s.d_v / kCombineCols)),
                         dim3(kCombineThreads), 0, stream, s.d_v, a2, m2, state_out);
      return check_launch("state combine launch");
    }
  }
  // with outputs and bf16 inputs, 16 columns per workgroup where even that grid fits
  constexpr bool kNarrow = FWD && sizeof(TIn) == 2;
  if constexpr (kNarrow) {
    if (2 * col_groups <= static_cast<uint32_t>(cus)) {
      hipLaunchKernelGGL((k_scan_cols<TIn, DK, FWD, 1>), dim3(2 * col_groups), dim3(cols_threads(FWD, false, 1)), 0,
                         stream, cu, s.num_k_heads, s.num_v_heads, s.d_v, static_cast<const TIn*>(v),
                         static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw, Tw, Sw, Pw, state_in,
                         static_cast<TIn*>(o), state_out);
      return check_launch("scan launch");
    }
  }
  // fp32 inputs with outputs: a grid that does not fit takes the 32-column scan
  // over as many rounds as it needs, longest first.  The whole-head kernel's
  // eight waves (two per SIMD) cannot hold fp32 operands and spill: at 3, 16
  // and 36 sequences of 32 heads (1024 tokens) its forward scan took 213, 642
  // and 1391 us against 113, 566 and 1233-1260 us in this form.
  constexpr bool kColsOut = FWD && sizeof(TIn) == 4;
  if (fits) {
    hipLaunchKernelGGL((k_scan_cols<TIn, DK, FWD>), dim3(col_groups), dim3(cols_threads(FWD, sizeof(TIn) == 4)), 0,
                       stream, cu, s.num_k_heads, s.num_v_heads, s.d_v, static_cast<const TIn*>(v),
                       static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw, Tw, Sw, Pw, state_in,
                       static_cast<TIn*>(o), state_out);
  } else if constexpr (kColsOut) {
    hipLaunchKernelGGL((k_scan_cols_out_ord<TIn, DK>), dim3(col_groups), dim3(cols_threads(true, true)), 0, stream,
                       cu, p.order, s.num_k_heads, s.num_v_heads, s.d_v, static_cast<const TIn*>(v),
                       static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw, Tw, Sw, Pw, state_in,
                       static_cast<TIn*>(o), state_out);
  } else if constexpr (kWide) {
    // A batch whose 64-column one-tile grid takes at most three rounds of the
    // chip (one workgroup per CU) runs in it: its chains finish a chunk in
    // ~1.45 us against ~3.9 us for a lone wide workgroup per CU (at 3, 8 and
    // 12 sequences of 32 heads: 178 -> 88, 196 -> 182, 283 -> 270 us).
    const int64_t groups64 = static_cast<int64_t>(s.num_seqs) * s.num_v_heads * (s.d_v / kSplitCols2);
    if (groups64 <= 3 * static_cast<int64_t>(cus)) {
      hipLaunchKernelGGL((k_scan_cols_64<TIn, DK>), dim3(static_cast<uint32_t>(groups64)),
                         dim3((kSplitCols2 / 16 + 1) * kWave), 0, stream, cu, p.order, s.num_k_heads, s.num_v_heads,
                         s.d_v, static_cast<const TIn*>(v), static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw,
                         Tw, Sw, state_out);
      return check_launch("scan launch");
    }
    // Otherwise a whole head per workgroup (128 columns, four compute waves)
    // where d_v allows, two workgroups per CU.  When the last round of that
    // grid would be partly empty and its sequences fit on the chip at one
    // 64-column workgroup per CU, those sequences (the shortest, in
    // longest-first order) run in the one-tile scan after it instead.
    constexpr int kCols = DV >= 128 ? 128 : 64;
    const int64_t per_seq = static_cast<int64_t>(s.num_v_heads) * (s.d_v / kCols);
    const int64_t rem = static_cast<int64_t>(s.num_seqs) * per_seq % (2 * static_cast<int64_t>(cus));
    int32_t peel = 0;
    if (rem > 0 && s.num_seqs <= kMaxOrderedSeqs) {
      peel = static_cast<int32_t>((rem + per_seq - 1) / per_seq);
      if (peel >= s.num_seqs || static_cast<int64_t>(peel) * s.num_v_heads * (s.d_v / kSplitCols2) > cus) peel = 0;
    }
    const int32_t n_wide = s.num_seqs - peel;
    hipLaunchKernelGGL((k_scan_cols_wide<TIn, DK, kCols>), dim3(static_cast<uint32_t>(n_wide * per_seq)),
                       dim3(cols_wide_threads(kCols)), 0, stream, cu, p.order, s.num_k_heads, s.num_v_heads, s.d_v,
                       static_cast<const TIn*>(v), static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw, Tw, Sw,
                       state_out);
    if (peel > 0) {
      if ((st = check_launch("scan launch")) != GDN_OK) return st;
      SeqOrder po;
      po.n = peel;
      for (int32_t i = 0; i < peel; ++i) po.seq[i] = p.order.n > 0 ? p.order.seq[n_wide + i] : n_wide + i;
      hipLaunchKernelGGL((k_scan_cols_64<TIn, DK>), dim3(static_cast<uint32_t>(peel) * s.num_v_heads *
                                                           (s.d_v / kSplitCols2)),
                         dim3((kSplitCols2 / 16 + 1) * kWave), 0, stream, cu, po, s.num_k_heads, s.num_v_heads, s.d_v,
                         static_cast<const TIn*>(v), static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw, Tw,
                         Sw, state_out);
    }
  } else {
    // a whole head per workgroup, one per CU.  With outputs, when the grid's
    // last round would be partly empty and its sequences (the shortest, in
    // longest-first order) fit in two rounds of the 32-column scan with
    // output waves, they run in that after the whole-head grid (12 and 36
    // sequences of 32 heads, 16 chunks: 216 -> 205 and 557 -> 545 us).
    int32_t peel = 0;
    if constexpr (FWD) {
      const int64_t rem = static_cast<int64_t>(s.num_seqs) * s.num_v_heads % cus;
      if (rem > 0 && s.num_seqs <= kMaxOrderedSeqs) {
        peel = static_cast<int32_t>((rem + s.num_v_heads - 1) / s.num_v_heads);
        if (peel >= s.num_seqs ||
            static_cast<int64_t>(peel) * s.num_v_heads * (s.d_v / kColsPerGroup) > 2 * static_cast<int64_t>(cus))
          peel = 0;
      }
    }
    const int32_t n_head = s.num_seqs - peel;
    hipLaunchKernelGGL((k_scan_head<TIn, DK, DV, FWD>), dim3(static_cast<uint32_t>(n_head) * s.num_v_heads),
                       dim3(head_threads(DV)), 0, stream, cu, p.order, s.num_k_heads, s.num_v_heads,
                       static_cast<const TIn*>(v), static_cast<const TIn*>(k), static_cast<const TIn*>(q), Kw, Tw, Sw,
                       Pw, state_in, static_cast<TIn*>(o), state_out);
    if constexpr (FWD) {
      if (peel > 0) {
        if ((st = check_launch("scan launch")) != GDN_OK) return st;
        SeqOrder po;
        po.n = peel;
        for (int32_t i = 0; i < peel; ++i) po.seq[i] = p.order.n > 0 ? p.order.seq[n_head + i] : n_head + i;
        hipLaunchKernelGGL((k_scan_cols_out_ord<TIn, DK>),
                           dim3(static_cast<uint32_t>(peel) * s.num_v_heads * (s.d_v / kColsPerGroup)),
                           dim3(cols_threads(true, sizeof(TIn) == 4)), 0, stream, cu, po, s.num_k_heads,
                           s.num_v_heads, s.d_v, static_cast<const TIn*>(v), static_cast<const TIn*>(k),
                           static_cast<const TIn*>(q), Kw, Tw, Sw, Pw, state_in, static_cast<TIn*>(o), state_out);
      }
    }
  }
  return check_launch("scan launch");
}

template <typename TIn, int DK, int DV, bool FWD>
gdn_status run(const Args& a) {
  const gdn_shape& s = *a.s;
  gdn_status st = mark(a, 0);
  if (st != GDN_OK) return st;
  if ((st = launch_intra<TIn, DK, FWD>(s, *a.p, a.cu, a.q, a.k, a.g, a.beta, a.ws, a.stream)) != GDN_OK)
    return st;
  if ((st = mark(a, 1)) != GDN_OK) return st;
  bool combined = false;
  if ((st = launch_scan<TIn, DK, DV, FWD>(s, *a.p, a.cu, a.v, a.k, a.q, a.state_in, a.o, a.state_out, a.ws,
                                          a.stream,
                                          FWD ? nullptr : &a, &combined)) != GDN_OK)
    return st;
  if (!FWD && !combined) {
    // one chain: the combine stage is empty
    if ((st = mark(a, 2)) != GDN_OK) return st;
  }
  return mark(a, num_stages(FWD));
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

gdn_status check_events(void* const* events, int32_t num_events, bool fwd) {
  if (!events) return fail(GDN_ERR_NULL_ARG, "stage_events is NULL");
  if (num_events != num_stages(fwd) + 1)
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
  if (shape->num_seqs == 0) return mark_all(a, false);
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
  if (shape->num_seqs == 0) return mark_all(a, true);
  return gdn::dispatch<true>(a);
}

// ---------------------------------------------------------------- replay then forward
constexpr int32_t kNumFusedStages = 4;
// The suffix's chunk preparation runs in the tail-scan stage when the tail is
// one chain (on the CUs the scan leaves idle) and in the combine stage when it
// runs in two halves (beside the combine); the combine stage is otherwise empty.
const char* const kFusedStageNames[kNumFusedStages] = {"tail intra", "tail scan (+ suffix intra)",
                                                       "combine (+ suffix intra)", "suffix scan"};

struct FusedArgs {
  const gdn_shape* s;
  const Plan* pt;      // tail plan (no outputs)
  const Plan* ps;      // suffix plan (outputs)
  const int32_t* cu_t;
  const void* k_t;
  const void* v_t;
  const float* g_t;
  const float* beta_t;
  const int32_t* cu_s;
  const void* q;
  const void* k;
  const void* v;
  const float* g;
  const float* beta;
  float* state_mid;
  void* o;
  float* state_out;
  char* ws_t;
  char* ws_s;
  hipStream_t stream;
  void* const* events;   // NULL, or kNumFusedStages + 1 events
};

gdn_status fmark(const FusedArgs& a, int stage) {
  if (!a.events) return GDN_OK;
  const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(a.events[stage]), a.stream);
  if (e != hipSuccess) return fail(GDN_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
  return GDN_OK;
}

template <typename TIn, int DK, int DV>
gdn_status run_fused(const FusedArgs& a) {
  const gdn_shape& s = *a.s;
  const Plan& pt = *a.pt;
  const Plan& ps = *a.ps;
  gdn_status st = fmark(a, 0);
  if (st != GDN_OK) return st;
  if ((st = launch_intra<TIn, DK, false>(s, pt, a.cu_t, nullptr, a.k_t, a.g_t, a.beta_t, a.ws_t, a.stream)) !=
      GDN_OK)
    return st;
  if ((st = fmark(a, 1)) != GDN_OK) return st;
  bool fits = false;
  uint32_t n_scan = 0;
  int cus = 0;
  if ((st = cols_fit(s, &fits, &n_scan, &cus)) != GDN_OK) return st;
  constexpr bool kCanSplit = sizeof(TIn) == 2;   // the split form is bf16 tail replay
  bool combine = false;
  if constexpr (kCanSplit) {
    if (pt.split && split_groups(s) <= cus && ps.num_slots > 0) {
      // the tail in two halves (as gdn_tail_replay runs it), then its combine
      // with the suffix's records built beside it
      hipLaunchKernelGGL((k_scan_cols_split<TIn, DK>), dim3(static_cast<uint32_t>(split_groups(s))),
                         dim3(cols_split_threads()), 0, a.stream,
                         static_cast<int32_t>(split_first_groups(s)), a.cu_t, s.num_k_heads, s.num_v_heads, s.d_v, static_cast<const TIn*>(a.v_t),
                         static_cast<const TIn*>(a.k_t), static_cast<const TIn*>(nullptr),
                         reinterpret_cast<const u32x4*>(a.ws_t + pt.off_K),
                         reinterpret_cast<const u32x4*>(a.ws_t + pt.off_T),
                         reinterpret_cast<const float*>(a.ws_t + pt.off_S), a.state_mid,
                         reinterpret_cast<float*>(a.ws_t + pt.off_M2), reinterpret_cast<float*>(a.ws_t + pt.off_A2));
      if ((st = check_launch("split scan launch")) != GDN_OK) return st;
      if ((st = fmark(a, 2)) != GDN_OK) return st;
      const uint32_t n_comb = static_cast<uint32_t>(s.num_seqs) * s.num_v_heads * (s.d_v / kCombineCols);
      const uint32_t blocks = n_comb + static_cast<uint32_t>(ps.num_slots) * s.num_v_heads;
      hipLaunchKernelGGL((k_combine_intra<TIn, DK>), dim3(blocks), dim3(kCombineThreads), 0, a.stream,
                         static_cast<int32_t>(n_comb), s.d_v, reinterpret_cast<const float*>(a.ws_t + pt.off_A2),
                         reinterpret_cast<const float*>(a.ws_t + pt.off_M2), a.state_mid,
                         static_cast<int32_t>(ps.num_slots), a.cu_s, s.num_seqs, s.num_k_heads, s.num_v_heads,
                         static_cast<const TIn*>(a.q), static_cast<const TIn*>(a.k), a.g, a.beta, s.scale,
                         reinterpret_cast<u32x4*>(a.ws_s + ps.off_K), reinterpret_cast<u32x4*>(a.ws_s + ps.off_T),
                         reinterpret_cast<float*>(a.ws_s + ps.off_S), reinterpret_cast<u32x4*>(a.ws_s + ps.off_P));
      if ((st = check_launch("combine + suffix intra launch")) != GDN_OK) return st;
      combine = true;
    }
  }
  if (!combine && fits && ps.num_slots > 0) {
    // the suffix's records are built on the CUs the tail replay leaves idle
    const uint32_t blocks = n_scan + static_cast<uint32_t>(ps.num_slots) * s.num_v_heads;
    hipLaunchKernelGGL((k_scan_cols_intra<TIn, DK>), dim3(blocks), dim3(4 * kWave), 0, a.stream,
                       static_cast<int32_t>(n_scan), a.cu_t, s.num_k_heads, s.num_v_heads, s.d_v,
                       static_cast<const TIn*>(a.v_t), static_cast<const TIn*>(a.k_t),
                       reinterpret_cast<const u32x4*>(a.ws_t + pt.off_K),
                       reinterpret_cast<const u32x4*>(a.ws_t + pt.off_T),
                       reinterpret_cast<const float*>(a.ws_t + pt.off_S), a.state_mid,
                       static_cast<int32_t>(ps.num_slots), a.cu_s, s.num_seqs, static_cast<const TIn*>(a.q),
                       static_cast<const TIn*>(a.k), a.g, a.beta, s.scale,
                       reinterpret_cast<u32x4*>(a.ws_s + ps.off_K), reinterpret_cast<u32x4*>(a.ws_s + ps.off_T),
                       reinterpret_cast<float*>(a.ws_s + ps.off_S), reinterpret_cast<u32x4*>(a.ws_s + ps.off_P));
    if ((st = check_launch("tail scan + suffix intra launch")) != GDN_OK) return st;
  } else if (!combine) {
    if ((st = launch_scan<TIn, DK, DV, false>(s, pt, a.cu_t, a.v_t, a.k_t, nullptr, nullptr, nullptr, a.state_mid,
                                              a.ws_t,
                                              a.stream)) != GDN_OK)
      return st;
    if ((st = launch_intra<TIn, DK, true>(s, ps, a.cu_s, a.q, a.k, a.g, a.beta, a.ws_s, a.stream)) != GDN_OK)
      return st;
  }
  if (!combine && (st = fmark(a, 2)) != GDN_OK) return st;
  if ((st = fmark(a, 3)) != GDN_OK) return st;
  if ((st = launch_scan<TIn, DK, DV, true>(s, ps, a.cu_s, a.v, a.k, a.q, a.state_mid, a.o, a.state_out, a.ws_s,
                                           a.stream)) != GDN_OK)
    return st;
  return fmark(a, 4);
}

template <int DK, int DV>
gdn_status fused_dtype(const FusedArgs& a) {
  return a.s->qkv_dtype == GDN_BF16 ? run_fused<uint16_t, DK, DV>(a) : run_fused<float, DK, DV>(a);
}

gdn_status fused_plans(const gdn_shape* shape, const int32_t* cu_tail_host, const int32_t* cu_suf_host,
                       Plan* pt, Plan* ps, size_t* off_s, size_t* bytes) {
  std::string err;
  gdn_status st = make_plan(shape, cu_tail_host, false, pt, &err);
  if (st != GDN_OK) return fail(st, "tail: " + err);
  if ((st = make_plan(shape, cu_suf_host, true, ps, &err)) != GDN_OK) return fail(st, "suffix: " + err);
  *off_s = (pt->bytes + kAlign - 1) / kAlign * kAlign;
  *bytes = *off_s + ps->bytes;
  return GDN_OK;
}

gdn_status replay_forward_impl(const gdn_shape* shape, const int32_t* cu_tail_host, const int32_t* cu_tail,
                               const void* k_tail, const void* v_tail, const float* g_tail,
                               const float* beta_tail, const int32_t* cu_suf_host, const int32_t* cu_suf,
                               const void* q, const void* k, const void* v, const float* g,
                               const float* beta, float* state_mid, void* o, float* state_out,
                               void* workspace, size_t workspace_bytes, void* stream, void* const* events) {
  Plan pt, ps;
  size_t off_s = 0, bytes = 0;
  gdn_status st = fused_plans(shape, cu_tail_host, cu_suf_host, &pt, &ps, &off_s, &bytes);
  if (st != GDN_OK) return st;
  if (shape->num_seqs > 0 && (!cu_tail || !cu_suf)) return fail(GDN_ERR_NULL_ARG, "cu_seqlens (device) is NULL");
  if (bytes > 0 && !workspace) return fail(GDN_ERR_WORKSPACE, "workspace is NULL");
  if (workspace_bytes < bytes)
    return fail(GDN_ERR_WORKSPACE, "workspace too small: need " + std::to_string(bytes) + " bytes, got " +
                                       std::to_string(workspace_bytes));
  if (reinterpret_cast<uintptr_t>(workspace) % kAlign != 0)
    return fail(GDN_ERR_WORKSPACE, "workspace must be 256-byte aligned");
  if (shape->num_seqs > 0 && !state_mid) return fail(GDN_ERR_NULL_ARG, "state_mid is NULL");
  if (pt.total_tokens > 0 && (!k_tail || !v_tail || !g_tail || !beta_tail))
    return fail(GDN_ERR_NULL_ARG, "k_tail, v_tail, g_tail and beta_tail must be non-NULL");
  if (ps.total_tokens > 0 && (!q || !k || !v || !g || !beta || !o))
    return fail(GDN_ERR_NULL_ARG, "q, k, v, g, beta and o must be non-NULL");
  for (const void* ptr : {k_tail, v_tail, q, k, v, static_cast<const void*>(o)})
    if (reinterpret_cast<uintptr_t>(ptr) % 16 != 0)
      return fail(GDN_ERR_UNSUPPORTED, "k_tail, v_tail, q, k, v and o must be 16-byte aligned");
  if (state_out && state_out != state_mid) {
    const size_t n = static_cast<size_t>(shape->num_seqs) * shape->num_v_heads * shape->d_k * shape->d_v;
    if (state_mid < state_out + n && state_out < state_mid + n)
      return fail(GDN_ERR_BAD_SHAPE, "state_out overlaps state_mid without being equal");
  }
  const FusedArgs a{shape, &pt, &ps, cu_tail, k_tail, v_tail, g_tail, beta_tail, cu_suf, q, k, v, g, beta,
                    state_mid, o, state_out, static_cast<char*>(workspace),
                    static_cast<char*>(workspace) + off_s, static_cast<hipStream_t>(stream), events};
  if (shape->num_seqs == 0) {
    for (int i = 0; i <= kNumFusedStages; ++i)
      if ((st = fmark(a, i)) != GDN_OK) return st;
    return GDN_OK;
  }
  const int dk = shape->d_k, dv = shape->d_v;
  if (dk == 64) return dv == 64 ? fused_dtype<64, 64>(a) : fused_dtype<64, 128>(a);
  return dv == 64 ? fused_dtype<128, 64>(a) : fused_dtype<128, 128>(a);
}

}  // namespace
}  // namespace gdn

namespace gdn {
namespace {

template <typename TIn, int DK, int DV>
void launch_decode(const gdn_shape& s, const void* q, const void* k, const void* v, const float* g,
                   const float* beta, const float* state_in, void* o, float* state_out, hipStream_t stream) {
  const uint32_t blocks = static_cast<uint32_t>(s.num_seqs) * s.num_v_heads;
  hipLaunchKernelGGL((k_decode<TIn, DK, DV>), dim3(blocks), dim3(kDecodeThreads), 0, stream, s.num_k_heads,
                     s.num_v_heads, static_cast<const TIn*>(q), static_cast<const TIn*>(k),
                     static_cast<const TIn*>(v), g, beta, s.scale, state_in, static_cast<TIn*>(o), state_out);
}

template <typename TIn>
void decode_dims(const gdn_shape& s, const void* q, const void* k, const void* v, const float* g,
                 const float* beta, const float* state_in, void* o, float* state_out, hipStream_t stream) {
  if (s.d_k == 64) {
    if (s.d_v == 64) launch_decode<TIn, 64, 64>(s, q, k, v, g, beta, state_in, o, state_out, stream);
    else launch_decode<TIn, 64, 128>(s, q, k, v, g, beta, state_in, o, state_out, stream);
  } else {
    if (s.d_v == 64) launch_decode<TIn, 128, 64>(s, q, k, v, g, beta, state_in, o, state_out, stream);
    else launch_decode<TIn, 128, 128>(s, q, k, v, g, beta, state_in, o, state_out, stream);
  }
}

gdn_status decode_step_impl(const gdn_shape* shape, const void* q, const void* k, const void* v,
                            const float* g, const float* beta, const float* state_in, void* o,
                            float* state_out, void* stream) {
  std::string err;
  const gdn_status st = check_shape(shape, &err);
  if (st != GDN_OK) return fail(st, err);
  if (shape->num_seqs == 0) return GDN_OK;
  if (!q || !k || !v || !g || !beta || !o || !state_out)
    return fail(GDN_ERR_NULL_ARG, "q, k, v, g, beta, o and state_out must be non-NULL");
  auto misaligned = [](const void* p) { return reinterpret_cast<uintptr_t>(p) % 16 != 0; };
  if (misaligned(q) || misaligned(k) || misaligned(v) || misaligned(o) || misaligned(state_out) ||
      (state_in && misaligned(state_in)))
    return fail(GDN_ERR_UNSUPPORTED, "q, k, v, o and the states must be 16-byte aligned");
  if (state_in && state_in != state_out) {
    const size_t n = static_cast<size_t>(shape->num_seqs) * shape->num_v_heads * shape->d_k * shape->d_v;
    if (state_in < state_out + n && state_out < state_in + n)
      return fail(GDN_ERR_BAD_SHAPE, "state_out overlaps state_in without being equal");
  }
  const hipStream_t s = static_cast<hipStream_t>(stream);
  if (shape->qkv_dtype == GDN_BF16) decode_dims<uint16_t>(*shape, q, k, v, g, beta, state_in, o, state_out, s);
  else decode_dims<float>(*shape, q, k, v, g, beta, state_in, o, state_out, s);
  return check_launch("decode launch");
}

}  // namespace
}  // namespace gdn

namespace gdn {
namespace {

// ---------------------------------------------------------------- replay without allocation
// Workspace of gdn_tail_replay_noalloc: a file-scope device array, one copy
// per GPU the library runs on, held until the process ends.  In host code
// `scratch` only names the symbol; its device address on each GPU comes from
// hipGetSymbolAddress on that GPU's first call and is kept per device.
constexpr size_t kNoAllocScratchBytes = size_t{GDN_NOALLOC_SCRATCH_BYTES};
static_assert(kNoAllocScratchBytes % kAlign == 0, "scratch size");
__device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// The scratch array's address on the current device.
gdn_status scratch_on_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(GDN_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxScratchDevices)
    return fail(GDN_ERR_UNSUPPORTED, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr)
      return fail(GDN_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    if (reinterpret_cast<uintptr_t>(ptr) % kAlign != 0)
      return fail(GDN_ERR_HIP, "scratch array is not 256-byte aligned");
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return GDN_OK;
}

gdn_status tail_replay_noalloc_impl(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                                    const int32_t* cu_seqlens, const void* k, const void* v, const float* g,
                                    const float* beta, float* state_out, void* stream) {
  // the plan first: an input too large for the scratch array is rejected
  // before anything touches the device
  Plan plan;
  std::string err;
  const gdn_status st = make_plan(shape, cu_seqlens_host, false, &plan, &err);
  if (st != GDN_OK) return fail(st, err);
  if (plan.bytes > kNoAllocScratchBytes)
    return fail(GDN_ERR_WORKSPACE, "input needs " + std::to_string(plan.bytes) +
                                       " workspace bytes, more than the no-allocation scratch array holds (" +
                                       std::to_string(kNoAllocScratchBytes) + ")");
  void* ws = nullptr;
  if (shape->num_seqs > 0 && plan.bytes > 0) {
    const gdn_status sst = scratch_on_current_device(&ws);
    if (sst != GDN_OK) return sst;
  }
  return tail_replay_impl(shape, cu_seqlens_host, cu_seqlens, k, v, g, beta, state_out, ws,
                          ws ? kNoAllocScratchBytes : 0, stream, nullptr);
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

gdn_status gdn_tail_replay_noalloc(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                                   const int32_t* cu_seqlens, const void* k, const void* v, const float* g,
                                   const float* beta, float* state_out, void* stream) {
  return gdn::tail_replay_noalloc_impl(shape, cu_seqlens_host, cu_seqlens, k, v, g, beta, state_out, stream);
}

size_t gdn_noalloc_scratch_bytes(void) { return gdn::kNoAllocScratchBytes; }

gdn_status gdn_tail_replay_profiled(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                                    const int32_t* cu_seqlens, const void* k, const void* v,
                                    const float* g, const float* beta, float* state_out,
                                    void* workspace, size_t workspace_bytes, void* stream,
                                    void* const* stage_events, int32_t num_events) {
  const gdn_status st = gdn::check_events(stage_events, num_events, false);
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
  const gdn_status st = gdn::check_events(stage_events, num_events, true);
  if (st != GDN_OK) return st;
  return gdn::chunk_forward_impl(shape, cu_seqlens_host, cu_seqlens, q, k, v, g, beta,
                                 state_in, o, state_out, workspace, workspace_bytes, stream,
                                 stage_events);
}

gdn_status gdn_replay_forward_workspace_size(const gdn_shape* shape, const int32_t* cu_tail_host,
                                             const int32_t* cu_suf_host, size_t* bytes) {
  if (!bytes) return gdn::fail(GDN_ERR_NULL_ARG, "bytes is NULL");
  gdn::Plan pt, ps;
  size_t off_s = 0;
  return gdn::fused_plans(shape, cu_tail_host, cu_suf_host, &pt, &ps, &off_s, bytes);
}

gdn_status gdn_replay_forward(const gdn_shape* shape, const int32_t* cu_tail_host, const int32_t* cu_tail,
                              const void* k_tail, const void* v_tail, const float* g_tail,
                              const float* beta_tail, const int32_t* cu_suf_host, const int32_t* cu_suf,
                              const void* q, const void* k, const void* v, const float* g, const float* beta,
                              float* state_mid, void* o, float* state_out, void* workspace,
                              size_t workspace_bytes, void* stream) {
  return gdn::replay_forward_impl(shape, cu_tail_host, cu_tail, k_tail, v_tail, g_tail, beta_tail, cu_suf_host,
                                  cu_suf, q, k, v, g, beta, state_mid, o, state_out, workspace, workspace_bytes,
                                  stream, nullptr);
}

gdn_status gdn_replay_forward_profiled(const gdn_shape* shape, const int32_t* cu_tail_host,
                                       const int32_t* cu_tail, const void* k_tail, const void* v_tail,
                                       const float* g_tail, const float* beta_tail, const int32_t* cu_suf_host,
                                       const int32_t* cu_suf, const void* q, const void* k, const void* v,
                                       const float* g, const float* beta, float* state_mid, void* o,
                                       float* state_out, void* workspace, size_t workspace_bytes, void* stream,
                                       void* const* stage_events, int32_t num_events) {
  if (!stage_events) return gdn::fail(GDN_ERR_NULL_ARG, "stage_events is NULL");
  if (num_events != gdn::kNumFusedStages + 1)
    return gdn::fail(GDN_ERR_BAD_SHAPE, "num_events must be gdn_replay_forward_num_stages() + 1");
  for (int i = 0; i < num_events; ++i)
    if (!stage_events[i]) return gdn::fail(GDN_ERR_NULL_ARG, "a stage event is NULL");
  return gdn::replay_forward_impl(shape, cu_tail_host, cu_tail, k_tail, v_tail, g_tail, beta_tail, cu_suf_host,
                                  cu_suf, q, k, v, g, beta, state_mid, o, state_out, workspace, workspace_bytes,
                                  stream, stage_events);
}

gdn_status gdn_decode_step(const gdn_shape* shape, const void* q, const void* k, const void* v,
                           const float* g, const float* beta, const float* state_in, void* o,
                           float* state_out, void* stream) {
  return gdn::decode_step_impl(shape, q, k, v, g, beta, state_in, o, state_out, stream);
}

int32_t gdn_replay_forward_num_stages(void) { return gdn::kNumFusedStages; }

const char* gdn_replay_forward_stage_name(int32_t stage) {
  if (stage < 0 || stage >= gdn::kNumFusedStages) return "";
  return gdn::kFusedStageNames[stage];
}

int32_t gdn_num_stages(int32_t with_outputs) { return gdn::num_stages(with_outputs != 0); }

const char* gdn_stage_name(int32_t with_outputs, int32_t stage) {
  if (stage < 0 || stage >= gdn::num_stages(with_outputs != 0)) return "";
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

const char* gdn_last_error(void) { return gdn::last_error(); }

}  // extern "C"
