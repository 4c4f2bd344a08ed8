// Plain bf16 GEMMs for the layer block's two projections, through hipBLASLt.
//
// Both projections are linear layers with weights stored [out_features,
// in_features] and activations token-major, so each is
//     D[n][m] = sum_k B[n][k] A[m][k]          (row-major D = B A^T)
// with A the weight [m, k] and B the activations [n, k].  In hipBLASLt's
// column-major terms that is D^T = A^T(op T) B^T(op N): the "TN" form.
// Inputs are bf16, accumulation fp32, D is bf16 or fp32.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>
#include <string>

#include "gdn_tail_replay.h"

namespace gdn {

// Row-major D [n, ldd] (first m columns) = B [n, ldb] (first k columns) times
// the transpose of A [m, lda] (first k columns).  d_dtype is GDN_BF16 or
// GDN_F32.  Enqueues on `stream`; returns GDN_ERR_HIP with a message when
// hipBLASLt fails or offers no algorithm.  The first call on a device creates
// that device's hipBLASLt handle (kept until the process ends); algorithm
// choices are cached per problem.  Thread-safe.
gdn_status gemm_tn(int64_t m, int64_t n, int64_t k, const void* a, int64_t lda, const void* b,
                   int64_t ldb, void* d, int64_t ldd, int32_t d_dtype, void* workspace,
                   size_t workspace_bytes, hipStream_t stream, std::string* err);

}  // namespace gdn
