/*
 * gdn_la_block.h -- C ABI of the linear-attention layer block replay in
 * libgdn_tailreplay.so (MI355X, gfx950).
 *
 * Tail-Replay feeds the cached full-attention output hiddens of the replayed
 * tail through each linear-attention layer of a group, which turns them into
 * the recurrence's k, v, alpha, beta (paper Section 3, Eq. 2); for the
 * group's last layer nothing but the rebuilt state is needed, so no output
 * path and no feed-forward block run for it.  The paper does not print the
 * layer; this is the Gated DeltaNet token mixer as such layers are usually
 * built, for T packed tokens (sequences by cu_seqlens):
 *
 *   1. P = X W_in^T, rows of W_in [q | k | v | a | b | z]
 *        (cq = Hk d_k, cq, cv = Hv d_v, Hv, Hv, cv rows);
 *   2. q, k, v = SiLU(causal depthwise conv, 4 taps, of their P columns),
 *        the convolution history zero before each sequence's first token
 *        (the replay starts the layer from scratch, like the state);
 *   3. q, k divided by sqrt(sum of squares + l2_eps) per (token, head);
 *   4. g = -exp(A_log) softplus(a + dt_bias), beta = sigmoid(b) per value head;
 *   5. Eq. 1 from the zero state (Eq. 2), o_t = scale S_t q_t;
 *   6. y = o / sqrt(mean(o^2) + norm_eps) * norm_w * silu(z) per (token, value head);
 *   7. out = Y W_out^T.
 *
 * Layouts (C-contiguous, token-major, device memory):
 *   x        [T, D]              bf16   the cached hiddens (the layer's input)
 *   w_in     [2cq + 2cv + 2Hv, D] bf16  linear-layer layout [out, in]
 *   conv_w   [2cq + cv, 4]       fp32   taps of the q | k | v channels; tap j
 *                                       multiplies token t - 3 + j (j = 3: t itself)
 *   a_log, dt_bias [Hv]          fp32
 *   norm_w   [d_v]               fp32   shared by the value heads
 *   w_out    [D, cv]             bf16   linear-layer layout
 *   state_out [N, Hv, d_k, d_v]  fp32   M = S^T, as in gdn_tail_replay.h
 *   out      [T, D]              bf16
 *
 * act_dtype sets the type of the intermediates between the kernels: the
 * in-projection P, the recurrence inputs q, k, v and its output o.  GDN_F32
 * keeps them in fp32 (the in-projection still multiplies bf16 by bf16 with
 * fp32 accumulation), so the block adds no rounding beyond the bf16 operands
 * of the out-projection; GDN_BF16 stores them in bf16, the precision such
 * layers usually run at, with half the intermediate traffic.
 *
 * Conventions as in gdn_tail_replay.h (caller-owned buffers and workspace,
 * host-side validation before anything is enqueued, everything on `stream`),
 * with two additions: the first call on a device creates that device's
 * hipBLASLt handle, kept until the process ends, and the matmul descriptors
 * and algorithm choice of each projection shape are cached with it (at most
 * 512 shapes; beyond that they are prepared per call) (the projections run
 * through hipBLASLt; their workspace is part of the caller's), and `out` may alias
 * `x` (x is read only by the in-projection, before out is written).  To
 * capture calls in a HIP graph, make one eager call of the same shape first
 * (the handle and the projections' algorithm choice are set up on it).
 * Requirements: D % 8 == 0, Hv % 4 == 0, d_k and d_v in {64, 128}, Hv % Hk == 0,
 * conv_taps == 4; x, w_in, w_out, out, conv_w and norm_w 16-byte aligned; workspace
 * 256-byte aligned.
 */
#ifndef GDN_LA_BLOCK_H
#define GDN_LA_BLOCK_H

#include "gdn_tail_replay.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t num_seqs;     /* N >= 0                                            */
  int32_t hidden;       /* D: model width, multiple of 8                     */
  int32_t num_k_heads;  /* Hk                                                */
  int32_t num_v_heads;  /* Hv, multiple of Hk and of 4                       */
  int32_t d_k;          /* 64 or 128                                         */
  int32_t d_v;          /* 64 or 128                                         */
  int32_t conv_taps;    /* 4                                                 */
  int32_t act_dtype;    /* gdn_dtype of the intermediates (see above)        */
  float scale;          /* o_t = scale S_t q_t                               */
  float l2_eps;         /* >= 0, inside the q/k norm                         */
  float norm_eps;       /* >= 0, inside the gated RMS norm                   */
} gdn_la_shape;

typedef struct {
  const void* w_in;     /* bf16 [2cq + 2cv + 2Hv, D]                          */
  const float* conv_w;  /* fp32 [2cq + cv, 4]                                 */
  const float* a_log;   /* fp32 [Hv]                                          */
  const float* dt_bias; /* fp32 [Hv]                                          */
  const float* norm_w;  /* fp32 [d_v]; may be NULL when out is NULL           */
  const void* w_out;    /* bf16 [D, cv]; may be NULL when out is NULL         */
} gdn_la_weights;

/*
 * Workspace bytes for gdn_la_block_replay with (with_outputs = 1) or without
 * (0) the block output.  Writes *bytes; returns a validation status.
 */
gdn_status gdn_la_block_workspace_size(const gdn_la_shape* shape,
                                       const int32_t* cu_seqlens_host,
                                       int32_t with_outputs, size_t* bytes);

/*
 * Replay of one linear-attention layer over the packed tails (paper Section 3,
 * Eq. 2 behind the layer's projections): steps 1-5 above write each
 * sequence's rebuilt state to state_out (required when N > 0); when `out` is
 * not NULL, steps 5-7 also write the layer output [T, D] (the next layer's
 * input); when it is NULL (a group's last layer) the query, z and output
 * paths are skipped and the in-projection computes only the k, v, a, b rows.
 * workspace: at least gdn_la_block_workspace_size(..., out != NULL) bytes.
 */
gdn_status gdn_la_block_replay(const gdn_la_shape* shape, const gdn_la_weights* weights,
                               const int32_t* cu_seqlens_host, const int32_t* cu_seqlens,
                               const void* x, float* state_out, void* out,
                               void* workspace, size_t workspace_bytes, void* stream);

/*
 * Profiling variant: identical work and results; records stage_events[i]
 * (hipEvent_t) before stage i and stage_events[n] after the last, where
 * n = gdn_la_block_num_stages(out != NULL) and num_events must be n + 1.
 */
gdn_status gdn_la_block_replay_profiled(const gdn_la_shape* shape, const gdn_la_weights* weights,
                                        const int32_t* cu_seqlens_host, const int32_t* cu_seqlens,
                                        const void* x, float* state_out, void* out,
                                        void* workspace, size_t workspace_bytes, void* stream,
                                        void* const* stage_events, int32_t num_events);

int32_t gdn_la_block_num_stages(int32_t with_outputs);
const char* gdn_la_block_stage_name(int32_t with_outputs, int32_t stage);

#ifdef __cplusplus
}
#endif

#endif /* GDN_LA_BLOCK_H */
