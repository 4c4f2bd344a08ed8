// Host-side validation and workspace planning for the GDN tail-replay library.
// Pure C++ (no HIP), so it can be built and sanitised on a machine without a GPU.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "gdn_tail_replay.h"

namespace gdn {

constexpr int kChunk = 64;        // tokens per chunk
constexpr size_t kAlign = 256;    // alignment of every workspace region

// Where each region lives inside the caller's workspace, and the launch sizes.
struct Plan {
  int64_t total_tokens = 0;
  int64_t num_chunks = 0;         // sum over sequences of ceil(len / 64)
  int32_t max_chunks = 0;         // longest sequence, in chunks
  bool with_outputs = false;
  // byte offsets into the workspace
  size_t off_seq_chunk = 0;       // int32 [N + 1]: first chunk of each sequence
  size_t off_chunk_info = 0;      // int32x2 [num_chunks]: (first token, length)
  size_t off_T = 0;               // fp32 [num_chunks, Hv, 64, 64]: (I + A)^-1
  size_t off_G = 0;               // fp32 [num_chunks, Hv, 64]: in-chunk cumulative log-gate
  size_t off_P = 0;               // fp32 [num_chunks, Hv, 64, 64]: scale * (Q K^T) * decay (outputs only)
  size_t bytes = 0;               // total workspace size
};

// Validates the shape and the host copy of the offsets and fills `plan`.
// Returns GDN_OK or a validation status with a message in `err`.
gdn_status make_plan(const gdn_shape* shape, const int32_t* cu_seqlens_host,
                     bool with_outputs, Plan* plan, std::string* err);

}  // namespace gdn
