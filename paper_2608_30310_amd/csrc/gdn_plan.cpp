// Host-side validation and workspace planning (see gdn_plan.h).
#include "gdn_plan.h"

#include <algorithm>
#include <cmath>
#include <limits>

namespace gdn {
namespace {

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

bool supported_dim(int32_t d) { return d == 64 || d == 128; }

constexpr int64_t kMaxGroups = std::numeric_limits<uint32_t>::max() / 256;

}  // namespace

namespace {
thread_local std::string t_last_error;
}  // namespace

void set_last_error(const std::string& msg) { t_last_error = msg; }
const char* last_error() { return t_last_error.c_str(); }

gdn_status check_shape(const gdn_shape* shape, std::string* err) {
  if (!shape) { *err = "shape is NULL"; return GDN_ERR_NULL_ARG; }
  const int32_t N = shape->num_seqs, hk = shape->num_k_heads, hv = shape->num_v_heads;
  if (N < 0) { *err = "num_seqs must be >= 0"; return GDN_ERR_BAD_SHAPE; }
  if (hk < 1 || hv < 1) { *err = "head counts must be >= 1"; return GDN_ERR_BAD_SHAPE; }
  if (hv % hk != 0) {
    *err = "num_v_heads must be a multiple of num_k_heads";
    return GDN_ERR_BAD_SHAPE;
  }
  if (shape->d_k < 1 || shape->d_v < 1) { *err = "head dimensions must be >= 1"; return GDN_ERR_BAD_SHAPE; }
  if (!supported_dim(shape->d_k) || !supported_dim(shape->d_v)) {
    *err = "d_k and d_v must each be 64 or 128";
    return GDN_ERR_UNSUPPORTED;
  }
  if (shape->qkv_dtype != GDN_F32 && shape->qkv_dtype != GDN_BF16) {
    *err = "qkv_dtype must be GDN_F32 or GDN_BF16";
    return GDN_ERR_UNSUPPORTED;
  }
  if (!std::isfinite(shape->scale)) { *err = "scale must be finite"; return GDN_ERR_BAD_SHAPE; }
  if (hv > 65535) { *err = "num_v_heads must be <= 65535"; return GDN_ERR_UNSUPPORTED; }
  // A grid dimension counts at most 2^32 - 1 work items; every kernel uses at
  // most 256 threads per workgroup and at most 4 workgroups per (sequence, head).
  if (static_cast<int64_t>(N) * hv * 4 > kMaxGroups) {
    *err = "num_seqs * num_v_heads too large";
    return GDN_ERR_UNSUPPORTED;
  }
  return GDN_OK;
}

gdn_status make_plan(const gdn_shape* shape, const int32_t* cu, bool with_outputs,
                     Plan* plan, std::string* err) {
  if (!plan) { *err = "plan is NULL"; return GDN_ERR_NULL_ARG; }
  const gdn_status st = check_shape(shape, err);
  if (st != GDN_OK) return st;
  const int32_t N = shape->num_seqs, hk = shape->num_k_heads, hv = shape->num_v_heads;
  if (!cu) { *err = "cu_seqlens_host is NULL"; return GDN_ERR_NULL_ARG; }
  if (cu[0] != 0) { *err = "cu_seqlens_host[0] must be 0"; return GDN_ERR_BAD_SEQLENS; }

  int64_t chunks = 0, slots = 0, prev_c = 0;
  int32_t max_chunks = 0;
  bool sorted = true;   // chunk counts non-increasing
  for (int32_t n = 0; n < N; ++n) {
    const int64_t len = static_cast<int64_t>(cu[n + 1]) - cu[n];
    if (len < 0) { *err = "cu_seqlens_host must be non-decreasing"; return GDN_ERR_BAD_SEQLENS; }
    const int64_t c = (len + kChunk - 1) / kChunk;
    if (n > 0 && c > prev_c) sorted = false;
    prev_c = c;
    chunks += c;
    if (c > 0) slots = std::max(slots, chunk_slot(cu[n], n) + c);
    if (c > max_chunks) max_chunks = static_cast<int32_t>(c);
  }
  const int64_t T = cu[N];
  // Units of work are addressed with 32-bit grid indices.
  if (chunks > std::numeric_limits<int32_t>::max() / 2) {
    *err = "too many chunks";
    return GDN_ERR_UNSUPPORTED;
  }
  if (slots > kMaxGroups) {
    *err = "too many chunk slots";
    return GDN_ERR_UNSUPPORTED;
  }

  Plan p;
  p.total_tokens = T;
  p.num_chunks = chunks;
  p.num_slots = slots;
  p.max_chunks = max_chunks;
  p.with_outputs = with_outputs;
  const size_t recs = static_cast<size_t>(slots) * hv;
  p.k_record = k_record_bytes(shape->d_k, with_outputs, shape->qkv_dtype == GDN_F32);
  size_t off = 0;
  p.off_K = off;
  off = align_up(off + p.k_record * static_cast<size_t>(slots) * hk);
  p.off_T = off;
  off = align_up(off + t_record_bytes(shape->qkv_dtype == GDN_F32) * recs);
  p.off_S = off;
  off = align_up(off + kSRecordBytes * recs);
  p.off_P = off;
  if (with_outputs) off = align_up(off + kPRecordBytes * recs);
  if (N >= 2 && N <= kMaxOrderedSeqs && !sorted) {
    int32_t idx[kMaxOrderedSeqs];
    for (int32_t n = 0; n < N; ++n) idx[n] = n;
    auto nch = [&](int32_t n) { return (static_cast<int64_t>(cu[n + 1]) - cu[n] + kChunk - 1) / kChunk; };
    std::stable_sort(idx, idx + N, [&](int32_t a, int32_t b) { return nch(a) > nch(b); });
    p.order.n = N;
    for (int32_t n = 0; n < N; ++n) p.order.seq[n] = idx[n];
  }
  p.split = !with_outputs && shape->qkv_dtype == GDN_BF16 && max_chunks >= kSplitMinChunks &&
            split_groups(*shape) <= kSplitMaxGroups;
  if (p.split) {
    const size_t heads = static_cast<size_t>(N) * hv;
    p.off_M2 = off;
    off = align_up(off + heads * shape->d_k * shape->d_v * sizeof(float));
    p.off_A2 = off;
    off = align_up(off + heads * shape->d_k * shape->d_k * sizeof(float));
  }
  p.bytes = off;
  *plan = p;
  return GDN_OK;
}

gdn_status make_block_plan(const gdn_la_shape* shape, const int32_t* cu, bool with_outputs,
                           BlockPlan* plan, std::string* err) {
  if (!plan) { *err = "plan is NULL"; return GDN_ERR_NULL_ARG; }
  if (!shape) { *err = "shape is NULL"; return GDN_ERR_NULL_ARG; }
  BlockPlan p;
  p.scan = gdn_shape{shape->num_seqs, shape->num_k_heads, shape->num_v_heads, shape->d_k,
                     shape->d_v, shape->act_dtype, shape->scale};
  gdn_status st = make_plan(&p.scan, cu, with_outputs, &p.scan_plan, err);
  if (st != GDN_OK) return st;
  const int32_t hk = shape->num_k_heads, hv = shape->num_v_heads;
  if (shape->hidden < 1) { *err = "hidden must be >= 1"; return GDN_ERR_BAD_SHAPE; }
  if (shape->hidden % 8 != 0) { *err = "hidden must be a multiple of 8"; return GDN_ERR_UNSUPPORTED; }
  if (shape->conv_taps != kBlockConvTaps) { *err = "conv_taps must be 4"; return GDN_ERR_UNSUPPORTED; }
  if (hv % 4 != 0) { *err = "num_v_heads must be a multiple of 4"; return GDN_ERR_UNSUPPORTED; }
  if (!std::isfinite(shape->l2_eps) || !std::isfinite(shape->norm_eps) || shape->l2_eps < 0.0f ||
      shape->norm_eps < 0.0f) {
    *err = "l2_eps and norm_eps must be finite and >= 0";
    return GDN_ERR_BAD_SHAPE;
  }
  p.T = p.scan_plan.total_tokens;
  p.outputs = with_outputs;
  p.cq = static_cast<int64_t>(hk) * shape->d_k;
  p.cv = static_cast<int64_t>(hv) * shape->d_v;
  const int64_t all_rows = 2 * p.cq + 2 * p.cv + 2 * hv;
  p.row0 = with_outputs ? 0 : p.cq;
  p.rows = with_outputs ? all_rows : p.cq + p.cv + 2 * hv;   // k | v | a | b
  p.ldp = p.rows;                                            // a multiple of 8 (Hv % 4 == 0)
  p.act_bytes = shape->act_dtype == GDN_F32 ? 4 : 2;
  const int64_t nch = with_outputs ? 2 * p.cq + p.cv : p.cq + p.cv;   // channels the prep computes
  p.prep_slabs = (nch + kBlockPrepChans - 1) / kBlockPrepChans + 1;
  // four tokens per thread once one-token units would fill the grid four
  // times over (measured at D = 2048: 3277 tokens 42.8 -> 37.1 us, while 819
  // tokens went 13.4 -> 14.6 us with too few units left to spread)
  const int64_t units1 = (p.T + kBlockPrepTokensPerThreadRow - 1) / kBlockPrepTokensPerThreadRow * p.prep_slabs;
  p.prep_tpt = units1 >= 4 * kBlockElementwiseGroups ? 4 : 1;
  const int64_t tokens_per_block = kBlockPrepTokensPerThreadRow * p.prep_tpt;
  p.prep_token_blocks = (p.T + tokens_per_block - 1) / tokens_per_block;
  p.norm_blocks = with_outputs ? (p.T * p.cv / 8 + 255) / 256 : 0;
  p.prep_grid = std::min(p.prep_token_blocks * p.prep_slabs, kBlockElementwiseGroups);
  p.norm_grid = std::min(p.norm_blocks, kBlockElementwiseGroups);
  if (p.T > std::numeric_limits<int32_t>::max() / 2 ||
      p.prep_token_blocks * p.prep_slabs > std::numeric_limits<int32_t>::max() ||
      p.norm_blocks > std::numeric_limits<int32_t>::max()) {
    *err = "too many tokens for one call";
    return GDN_ERR_UNSUPPORTED;
  }
  const size_t T = static_cast<size_t>(p.T), es = p.act_bytes;
  size_t off = 0;
  auto take = [&](size_t bytes) { const size_t at = off; off = align_up(off + bytes); return at; };
  p.off_P = take(T * p.ldp * es);
  p.off_q = with_outputs ? take(T * p.cq * es) : 0;
  p.off_k = take(T * p.cq * es);
  p.off_v = take(T * p.cv * es);
  p.off_g = take(T * hv * 4);
  p.off_beta = take(T * hv * 4);
  p.off_o = with_outputs ? take(T * p.cv * es) : 0;
  p.off_scan = take(p.scan_plan.bytes);
  p.off_gemm = take(kGemmWorkspace);
  p.bytes = off;
  *plan = p;
  return GDN_OK;
}

}  // namespace gdn
