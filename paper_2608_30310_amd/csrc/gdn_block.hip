// The linear-attention layer block replay (C ABI in gdn_la_block.h): the
// layer's projections and activations around the recurrence (paper Section 3,
// Eq. 2 fed by the layer's k, v, alpha, beta).
//
// Stages, all on the caller's stream:
//   in-projection   hipBLASLt bf16 GEMM, P = X W_in^T (only the k, v, a, b
//                   rows when no output is wanted)
//   prep            k_la_prep: conv + SiLU + L2 norms + gates (gdn_block.h)
//   recurrence      gdn_chunk_forward from the zero state (with outputs) or
//                   gdn_tail_replay (state only)
//   gated norm      k_gated_norm -> y bf16
//   out-projection  hipBLASLt bf16 GEMM, out = Y W_out^T
#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>

#include "gdn_block.h"
#include "gdn_gemm.h"
#include "gdn_la_block.h"
#include "gdn_plan.h"

namespace gdn {
namespace {

static_assert(prep_tokens(1) == kBlockPrepTokensPerThreadRow && kPrepChans == kBlockPrepChans &&
                  kConvTaps == kBlockConvTaps,
              "host and device tiling agree");

constexpr int32_t kBlockStagesOut = 5;
constexpr int32_t kBlockStagesState = 3;
const char* const kBlockStageNamesOut[kBlockStagesOut] = {"in-projection", "prep", "recurrence",
                                                          "gated norm", "out-projection"};
const char* const kBlockStageNamesState[kBlockStagesState] = {"in-projection", "prep", "recurrence"};

gdn_status bfail(gdn_status st, const std::string& msg) {
  set_last_error(msg);
  return st;
}

struct Marks {
  void* const* events;
  hipStream_t stream;
  gdn_status at(int stage) const {
    if (!events) return GDN_OK;
    const hipError_t e = hipEventRecord(static_cast<hipEvent_t>(events[stage]), stream);
    if (e != hipSuccess) return bfail(GDN_ERR_HIP, std::string("hipEventRecord: ") + hipGetErrorString(e));
    return GDN_OK;
  }
};

template <typename TA, int DK, int DV>
void launch_prep(const BlockPlan& p, const gdn_la_shape& s, const gdn_la_weights& w, const int32_t* cu,
                 char* ws, hipStream_t stream) {
  const uint32_t blocks = static_cast<uint32_t>(p.prep_grid);
  TA* q = p.outputs ? reinterpret_cast<TA*>(ws + p.off_q) : nullptr;
  auto kernel = p.prep_tpt == 4 ? k_la_prep<TA, TA, DK, DV, 4> : k_la_prep<TA, TA, DK, DV, 1>;
  hipLaunchKernelGGL(kernel, dim3(blocks), dim3(kPrepThreads), 0, stream,
                     static_cast<int32_t>(p.T), s.num_seqs, cu, s.num_k_heads, s.num_v_heads,
                     reinterpret_cast<const TA*>(ws + p.off_P), p.ldp,
                     static_cast<int32_t>(p.outputs ? 0 : p.cq), static_cast<int32_t>(p.prep_slabs - 1),
                     static_cast<int32_t>(p.prep_token_blocks), w.conv_w, w.a_log, w.dt_bias, s.l2_eps, q,
                     reinterpret_cast<TA*>(ws + p.off_k), reinterpret_cast<TA*>(ws + p.off_v),
                     reinterpret_cast<float*>(ws + p.off_g), reinterpret_cast<float*>(ws + p.off_beta));
}

template <typename TA, int DV>
void launch_norm(const BlockPlan& p, const gdn_la_shape& s, const gdn_la_weights& w, char* ws,
                 hipStream_t stream) {
  const int64_t groups = p.T * p.cv / 8;
  const int32_t col_z = static_cast<int32_t>(2 * p.cq + p.cv + 2 * s.num_v_heads);
  hipLaunchKernelGGL((k_gated_norm<TA, TA, DV>), dim3(static_cast<uint32_t>(p.norm_grid)),
                     dim3(kNormThreads), 0, stream, groups, static_cast<int32_t>(p.cv),
                     reinterpret_cast<const TA*>(ws + p.off_o), reinterpret_cast<const TA*>(ws + p.off_P),
                     p.ldp, col_z, w.norm_w, s.norm_eps, reinterpret_cast<uint16_t*>(ws + p.off_q));
}

template <typename TA>
void prep_dims(const BlockPlan& p, const gdn_la_shape& s, const gdn_la_weights& w, const int32_t* cu,
               char* ws, hipStream_t stream) {
  if (s.d_k == 64) {
    if (s.d_v == 64) launch_prep<TA, 64, 64>(p, s, w, cu, ws, stream);
    else launch_prep<TA, 64, 128>(p, s, w, cu, ws, stream);
  } else {
    if (s.d_v == 64) launch_prep<TA, 128, 64>(p, s, w, cu, ws, stream);
    else launch_prep<TA, 128, 128>(p, s, w, cu, ws, stream);
  }
}

template <typename TA>
void norm_dims(const BlockPlan& p, const gdn_la_shape& s, const gdn_la_weights& w, char* ws,
               hipStream_t stream) {
  if (s.d_v == 64) launch_norm<TA, 64>(p, s, w, ws, stream);
  else launch_norm<TA, 128>(p, s, w, ws, stream);
}

gdn_status launched(const char* what) {
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return bfail(GDN_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return GDN_OK;
}

bool misaligned(const void* p, size_t a) { return reinterpret_cast<uintptr_t>(p) % a != 0; }

gdn_status block_impl(const gdn_la_shape* shape, const gdn_la_weights* w, const int32_t* cu_host,
                      const int32_t* cu, const void* x, float* state_out, void* out, void* workspace,
                      size_t workspace_bytes, void* stream_ptr, void* const* events, int32_t num_events) {
  const bool outputs = out != nullptr;
  BlockPlan p;
  std::string err;
  gdn_status st = make_block_plan(shape, cu_host, outputs, &p, &err);
  if (st != GDN_OK) return bfail(st, err);
  if (events) {
    const int32_t want = (outputs ? kBlockStagesOut : kBlockStagesState) + 1;
    if (num_events != want) return bfail(GDN_ERR_BAD_SHAPE, "num_events must be gdn_la_block_num_stages() + 1");
    for (int i = 0; i < num_events; ++i)
      if (!events[i]) return bfail(GDN_ERR_NULL_ARG, "a stage event is NULL");
  }
  if (!w) return bfail(GDN_ERR_NULL_ARG, "weights is NULL");
  if (!w->w_in || !w->conv_w || !w->a_log || !w->dt_bias)
    return bfail(GDN_ERR_NULL_ARG, "w_in, conv_w, a_log and dt_bias must be non-NULL");
  if (outputs && (!w->norm_w || !w->w_out))
    return bfail(GDN_ERR_NULL_ARG, "norm_w and w_out must be non-NULL when out is given");
  if (shape->num_seqs > 0 && !state_out) return bfail(GDN_ERR_NULL_ARG, "state_out is NULL");
  if (shape->num_seqs > 0 && !cu) return bfail(GDN_ERR_NULL_ARG, "cu_seqlens (device) is NULL");
  if (p.T > 0 && !x) return bfail(GDN_ERR_NULL_ARG, "x is NULL");
  if (misaligned(x, 16) || misaligned(w->w_in, 16) || misaligned(w->conv_w, 16) ||
      (outputs && (misaligned(w->w_out, 16) || misaligned(w->norm_w, 16) || misaligned(out, 16))))
    return bfail(GDN_ERR_UNSUPPORTED, "x, w_in, conv_w, norm_w, w_out and out must be 16-byte aligned");
  if (!workspace) return bfail(GDN_ERR_WORKSPACE, "workspace is NULL");
  if (workspace_bytes < p.bytes)
    return bfail(GDN_ERR_WORKSPACE, "workspace too small: need " + std::to_string(p.bytes) + " bytes, got " +
                                        std::to_string(workspace_bytes));
  if (misaligned(workspace, kAlign)) return bfail(GDN_ERR_WORKSPACE, "workspace must be 256-byte aligned");

  const hipStream_t stream = static_cast<hipStream_t>(stream_ptr);
  const Marks mk{events, stream};
  char* ws = static_cast<char*>(workspace);
  const int64_t D = shape->hidden;
  const bool f32 = shape->act_dtype == GDN_F32;

  // 1. in-projection
  if ((st = mk.at(0)) != GDN_OK) return st;
  const uint16_t* w_in = static_cast<const uint16_t*>(w->w_in) + p.row0 * D;
  st = gemm_tn(p.rows, p.T, D, w_in, D, x, D, ws + p.off_P, p.ldp, shape->act_dtype, ws + p.off_gemm,
               kGemmWorkspace, stream, &err);
  if (st != GDN_OK) return bfail(st, "in-projection: " + err);
  // 2. conv, SiLU, norms, gates
  if ((st = mk.at(1)) != GDN_OK) return st;
  if (p.T > 0) {
    if (f32) prep_dims<float>(p, *shape, *w, cu, ws, stream);
    else prep_dims<uint16_t>(p, *shape, *w, cu, ws, stream);
    if ((st = launched("prep launch")) != GDN_OK) return st;
  }
  // 3. the recurrence from the zero state
  if ((st = mk.at(2)) != GDN_OK) return st;
  if (outputs) {
    st = gdn_chunk_forward(&p.scan, cu_host, cu, ws + p.off_q, ws + p.off_k, ws + p.off_v,
                           reinterpret_cast<const float*>(ws + p.off_g),
                           reinterpret_cast<const float*>(ws + p.off_beta), nullptr, ws + p.off_o, state_out,
                           ws + p.off_scan, p.scan_plan.bytes, stream);
  } else {
    st = gdn_tail_replay(&p.scan, cu_host, cu, ws + p.off_k, ws + p.off_v,
                         reinterpret_cast<const float*>(ws + p.off_g),
                         reinterpret_cast<const float*>(ws + p.off_beta), state_out, ws + p.off_scan,
                         p.scan_plan.bytes, stream);
  }
  if (st != GDN_OK) return st;   // the recurrence set the message
  if (!outputs) return mk.at(3);
  // 4. gated RMS norm -> y (bf16, over the consumed q | k | v region)
  if ((st = mk.at(3)) != GDN_OK) return st;
  if (p.T > 0) {
    if (f32) norm_dims<float>(p, *shape, *w, ws, stream);
    else norm_dims<uint16_t>(p, *shape, *w, ws, stream);
    if ((st = launched("gated norm launch")) != GDN_OK) return st;
  }
  // 5. out-projection
  if ((st = mk.at(4)) != GDN_OK) return st;
  st = gemm_tn(D, p.T, p.cv, w->w_out, p.cv, ws + p.off_q, p.cv, out, D, GDN_BF16, ws + p.off_gemm,
               kGemmWorkspace, stream, &err);
  if (st != GDN_OK) return bfail(st, "out-projection: " + err);
  return mk.at(5);
}

}  // namespace
}  // namespace gdn

extern "C" {

gdn_status gdn_la_block_workspace_size(const gdn_la_shape* shape, const int32_t* cu_seqlens_host,
                                       int32_t with_outputs, size_t* bytes) {
  if (!bytes) return gdn::bfail(GDN_ERR_NULL_ARG, "bytes is NULL");
  gdn::BlockPlan p;
  std::string err;
  const gdn_status st = gdn::make_block_plan(shape, cu_seqlens_host, with_outputs != 0, &p, &err);
  if (st != GDN_OK) return gdn::bfail(st, err);
  *bytes = p.bytes;
  return GDN_OK;
}

gdn_status gdn_la_block_replay(const gdn_la_shape* shape, const gdn_la_weights* weights,
                               const int32_t* cu_seqlens_host, const int32_t* cu_seqlens, const void* x,
                               float* state_out, void* out, void* workspace, size_t workspace_bytes,
                               void* stream) {
  return gdn::block_impl(shape, weights, cu_seqlens_host, cu_seqlens, x, state_out, out, workspace,
                         workspace_bytes, stream, nullptr, 0);
}

gdn_status gdn_la_block_replay_profiled(const gdn_la_shape* shape, const gdn_la_weights* weights,
                                        const int32_t* cu_seqlens_host, const int32_t* cu_seqlens,
                                        const void* x, float* state_out, void* out, void* workspace,
                                        size_t workspace_bytes, void* stream, void* const* stage_events,
                                        int32_t num_events) {
  if (!stage_events) return gdn::bfail(GDN_ERR_NULL_ARG, "stage_events is NULL");
  return gdn::block_impl(shape, weights, cu_seqlens_host, cu_seqlens, x, state_out, out, workspace,
                         workspace_bytes, stream, stage_events, num_events);
}

int32_t gdn_la_block_num_stages(int32_t with_outputs) {
  return with_outputs ? gdn::kBlockStagesOut : gdn::kBlockStagesState;
}

const char* gdn_la_block_stage_name(int32_t with_outputs, int32_t stage) {
  const int32_t n = gdn_la_block_num_stages(with_outputs);
  if (stage < 0 || stage >= n) return "";
  return with_outputs ? gdn::kBlockStageNamesOut[stage] : gdn::kBlockStageNamesState[stage];
}

}  // extern "C"
