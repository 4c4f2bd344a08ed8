// Host-side validation and workspace planning for the GDN tail-replay library.
// Pure C++ (no HIP), so it can be built and sanitised on a machine without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "gdn_la_block.h"
#include "gdn_tail_replay.h"

namespace gdn {

constexpr int kChunk = 64;        // tokens per chunk
constexpr size_t kAlign = 256;    // alignment of every workspace region

// Chunk j of sequence n uses workspace slot cu[n] / 64 + n + j.  The map is
// injective (ceil(len / 64) <= len / 64 + 1), so kernels find their records
// from cu_seqlens alone; at most N slots stay unused.
inline int64_t chunk_slot(int64_t seq_start, int64_t seq) { return seq_start / kChunk + seq; }

// Workspace records.  A fragment is one MFMA operand for a whole wave: 64 lanes
// x 8 bf16 = 1 KiB.  Per (slot, value head), T and P keep their six nonzero
// fragments and S the per-row scalars.  P is split into hi + lo parts; so is T
// for fp32 inputs, while for bf16 inputs the scan multiplies by hi(T) alone
// (the state's error stays below about 5e-4 relative, measured on the CPU with
// a model of the kernels' rounding), so the record holds hi(T) only.  The
// scan holds each chunk's keys in LDS as A operands for K M (4 row tiles x
// d_k/32 k steps; lane (g, r) of fragment (ti, kk) holds K[16 ti + r][32 kk +
// 8 g + j], j = 0..7, sixteen consecutive bytes of a key row) and, with
// outputs, the queries in the same form for Q M; it takes the operands of K^T
// Delta from the same fragments with transposing LDS reads.  For bf16 inputs
// those fragments are the input rows themselves, fetched by the scan's DMA;
// for fp32 inputs, which need hi and lo parts, the chunk preparation writes
// them as a K record per (slot, key head).
constexpr size_t kFragBytes = 1024;
constexpr int kTFrags = 6;                                   // nonzero (row tile, k step) pairs
constexpr size_t kPRecordBytes = 2 * kTFrags * kFragBytes;   // P, split hi/lo
constexpr int t_record_parts(bool split) { return split ? 2 : 1; }   // T: hi (and lo)
constexpr size_t t_record_bytes(bool split) { return t_record_parts(split) * kTFrags * kFragBytes; }
constexpr size_t kSRecordBytes = 5 * 64 * 4;                 // per-row fp32 scalars

constexpr int ka_frags(int dk) { return 4 * (dk / 32); }     // K as A for K M
constexpr int k_record_frags(int dk, bool outputs) {          // per bf16 part
  return ka_frags(dk) + (outputs ? ka_frags(dk) : 0);
}
// the chunk's K (and Q) fragments in the scan's LDS
constexpr size_t k_tile_bytes(int dk, bool outputs, bool split) {
  return static_cast<size_t>(k_record_frags(dk, outputs)) * (split ? 2 : 1) * kFragBytes;
}
// the K record in the workspace: fp32 inputs only
constexpr size_t k_record_bytes(int dk, bool outputs, bool split) {
  return split ? k_tile_bytes(dk, outputs, split) : 0;
}

// Longest-first order of a batch's sequences by chunk count (equal counts keep
// their index order): seq[r] = the sequence of rank r.  n = 0 means the
// identity: batches of one sequence, of more than kMaxOrderedSeqs, or whose
// chunk counts never rise.  Travels by value in a kernel's arguments.
constexpr int32_t kMaxOrderedSeqs = 256;
struct SeqOrder {
  int32_t n = 0;
  int32_t seq[kMaxOrderedSeqs];
};

// Where each region lives inside the caller's workspace, and the launch sizes.
struct Plan {
  int64_t total_tokens = 0;
  int64_t num_chunks = 0;         // sum over sequences of ceil(len / 64)
  int64_t num_slots = 0;          // 1 + largest slot index in use (0 if none)
  int32_t max_chunks = 0;         // longest sequence, in chunks
  bool with_outputs = false;
  size_t k_record = 0;            // bytes of one K record
  // byte offsets into the workspace
  size_t off_K = 0;               // [num_slots, Hk] K records
  size_t off_T = 0;               // [num_slots, Hv] T = (I + A)^-1 fragments
  size_t off_S = 0;               // [num_slots, Hv] row scalars
  size_t off_P = 0;               // [num_slots, Hv] P fragments (outputs only)
  // Longest-first order of the sequences, for scans whose grid exceeds the
  // chip (passed by value in the kernel's arguments)
  SeqOrder order;
  // Tail replay in two halves (see split_groups): the second half's state
  // from zero and its transition, fp32
  bool split = false;
  size_t off_M2 = 0;              // [N, Hv, d_k, d_v]
  size_t off_A2 = 0;              // [N, Hv, d_k, d_k]
  size_t bytes = 0;               // total workspace size
};

// Tail replay of bf16 inputs may run as two half-length scans and a combine
// when every workgroup of the split grid fits on the chip at once (one per CU):
// N x Hv x (d_v / 32 + (d_v + d_k) / 64) of them, at most kSplitMaxGroups (the
// MI355X's 256 CUs; fewer on a smaller device are checked at launch), and
// the longest sequence has at least kSplitMinChunks chunks.  Measured on
// MI355X: one chain of n chunks takes ~1.63 n + 2 us, the split ~1.06 n + 9.4
// (its chunks are slower with every CU busy, and the combine with the kernel
// boundary before it costs ~7 us), even at n = 13 and ahead beyond.
constexpr int64_t kSplitMaxGroups = 256;

constexpr int32_t kSplitMinChunks = 20;
// state columns per workgroup of the first and of the second half
constexpr int kSplitCols1 = 32, kSplitCols2 = 64;
inline int64_t split_first_groups(const gdn_shape& s) {
  return static_cast<int64_t>(s.num_seqs) * s.num_v_heads * (s.d_v / kSplitCols1);
}
inline int64_t split_groups(const gdn_shape& s) {
  return split_first_groups(s) +
         static_cast<int64_t>(s.num_seqs) * s.num_v_heads * ((s.d_v + s.d_k) / kSplitCols2);
}

// ---------------------------------------------------------------- layer block
// Workspace the two projections may use (hipBLASLt's split-k kernels).
constexpr size_t kGemmWorkspace = size_t{32} << 20;
constexpr int kBlockConvTaps = 4;
// tokens per prep workgroup: 8 x (tokens per thread, 1 or 4: prep_tokens on the device)
constexpr int kBlockPrepTokensPerThreadRow = 8;
constexpr int kBlockPrepChans = 256;  // channels per prep workgroup (kPrepChans)
// Grid cap of the two elementwise kernels: 8 workgroups of 256 threads per CU
// of the 256-CU MI355X (a multiple of 8, one per XCD); they stride over the rest.
constexpr int64_t kBlockElementwiseGroups = 2048;

// Regions of the layer block's workspace and the in-projection's extent.  P
// holds rows row0 .. row0 + rows of W_in applied to every token, pitch ldp.
// With outputs, y (bf16 [T, cv]) reuses the q | k | v region once the
// recurrence has consumed it.
struct BlockPlan {
  gdn_shape scan{};       // the recurrence's shape (qkv_dtype = act_dtype)
  Plan scan_plan;         // and its workspace plan
  int64_t T = 0;
  bool outputs = false;
  int64_t cq = 0, cv = 0;
  int64_t row0 = 0, rows = 0, ldp = 0;
  size_t act_bytes = 0;
  size_t off_P = 0, off_q = 0, off_k = 0, off_v = 0, off_g = 0, off_beta = 0, off_o = 0;
  size_t off_scan = 0, off_gemm = 0, bytes = 0;
  int32_t prep_tpt = 1;                            // tokens per prep thread (1 or 4)
  int64_t prep_token_blocks = 0, prep_slabs = 0;   // channel slabs, plus one gate slab
  int64_t prep_grid = 0;                            // workgroups launched (<= units)
  int64_t norm_blocks = 0, norm_grid = 0;
};

// Validates a layer-block call's shape and offsets and fills `plan`.
gdn_status make_block_plan(const gdn_la_shape* shape, const int32_t* cu_seqlens_host,
                           bool with_outputs, BlockPlan* plan, std::string* err);

// The thread-local message behind gdn_last_error(), shared by every entry point.
void set_last_error(const std::string& msg);
const char* last_error();

// Validates the shape alone (dimensions, dtype, scale, grid limits).
gdn_status check_shape(const gdn_shape* shape, std::string* err);

// Validates the shape and the host copy of the offsets and fills `plan`.
// Returns GDN_OK or a validation status with a message in `err`.
gdn_status make_plan(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                     bool with_outputs, Plan* plan, std::string* err);

}  // namespace gdn
