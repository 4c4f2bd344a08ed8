/*
 * gdn_tail_replay.h -- C ABI of the MI355X (gfx950) Gated DeltaNet
 * tail-replay library (libgdn_tailreplay.so).
 *
 * The operation (paper Section 2, Eq. 1; Section 3, Eq. 2).  For every packed
 * sequence n and value head h, with key/query head kh = h / (Hv / Hk), the
 * gated delta rule
 *     S_t = S_{t-1} alpha_t (I - beta_t k_t k_t^T) + beta_t v_t k_t^T,
 *     alpha_t = exp(g_t),
 * is applied token by token.  The state is stored transposed, M = S^T, as a
 * d_k x d_v row-major fp32 matrix (d_v fastest):
 *     M_t = alpha_t M_{t-1} + k_t (beta_t (v_t - alpha_t M_{t-1}^T k_t))^T.
 * Independent Tail-Replay (Eq. 2) starts from a zero state at the first token
 * of the replayed tail and keeps the state after its last token.  The forward
 * call continues from a given state and also emits o_t = scale * S_t q_t
 * (computed after the update of token t).
 *
 * Layouts (all buffers C-contiguous, tokens packed varlen, token-major):
 *     q, k     [T, Hk, d_k]        qkv_dtype
 *     v, o     [T, Hv, d_v]        qkv_dtype
 *     g, beta  [T, Hv]             fp32; g = log alpha <= 0, beta in [0, 1]
 *     state    [N, Hv, d_k, d_v]   fp32, M = S^T
 *     cu_seqlens [N + 1]           int32 token offsets, cu[0] = 0, cu[N] = T
 *
 * Conventions
 *   - Pointers are device pointers unless their name ends in _host.
 *   - The caller owns every buffer, including the workspace.  The library
 *     never allocates, never synchronises and never copies between host and
 *     device; every call only enqueues kernels on `stream` (a hipStream_t,
 *     NULL = the null stream) and returns.
 *   - Validation happens on the host, from cu_seqlens_host, before anything is
 *     enqueued; a rejected call launches nothing and writes nothing.  The
 *     caller guarantees that cu_seqlens (device) holds the same values.
 *   - g <= 0 and beta in [0, 1] are assumed, not checked.  q and k are used as
 *     given (normalising them is the caller's job).
 *   - Zero-length sequences are allowed: tail replay writes a zero state,
 *     forward writes state_in (or zeros when state_in is NULL).
 *   - q, k, v and o must be 16-byte aligned (GDN_ERR_UNSUPPORTED otherwise); the
 *     workspace 256-byte aligned (GDN_ERR_WORKSPACE otherwise).
 *   - Inputs are never written.  state_out may alias state_in only when the two
 *     pointers are equal.  Calls that share a workspace must be ordered on one
 *     stream.
 *   - Reentrant; the only global state is a thread-local error message.
 */
#ifndef GDN_TAIL_REPLAY_H
#define GDN_TAIL_REPLAY_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GDN_OK = 0,
  GDN_ERR_NULL_ARG = 1,     /* a required pointer is NULL                    */
  GDN_ERR_BAD_SHAPE = 2,    /* head counts / dimensions inconsistent         */
  GDN_ERR_BAD_SEQLENS = 3,  /* cu_seqlens_host not 0-based non-decreasing    */
  GDN_ERR_UNSUPPORTED = 4,  /* valid but not built: d not in {64,128}, dtype */
  GDN_ERR_WORKSPACE = 5,    /* workspace NULL or smaller than required       */
  GDN_ERR_HIP = 6           /* a HIP runtime call failed; see gdn_last_error */
} gdn_status;

typedef enum { GDN_F32 = 0, GDN_BF16 = 1 } gdn_dtype;

typedef struct {
  int32_t num_seqs;     /* N >= 0                                            */
  int32_t num_k_heads;  /* Hk >= 1: heads of q and k                         */
  int32_t num_v_heads;  /* Hv >= 1: heads of v, g, beta, o, state; Hv % Hk == 0 */
  int32_t d_k;          /* key head dimension, 64 or 128                     */
  int32_t d_v;          /* value head dimension, 64 or 128                   */
  int32_t qkv_dtype;    /* gdn_dtype of q, k, v and o                        */
  float scale;          /* output scale: o_t = scale * S_t q_t               */
} gdn_shape;

/*
 * Workspace bytes needed by gdn_tail_replay (with_outputs = 0) or
 * gdn_chunk_forward (with_outputs = 1) for this shape and these sequence
 * lengths.  Writes *bytes; returns a validation status (nothing enqueued).
 */
gdn_status gdn_workspace_size(const gdn_shape* shape,
                              const int32_t* cu_seqlens_host,
                              int32_t with_outputs, size_t* bytes);

/*
 * Independent Tail-Replay (paper Section 3, Eq. 2): for each sequence (one
 * replayed tail of a matched prefix, packed by cu_seqlens) and value head,
 * start from the zero state and apply Eq. 1 to every token; write the state
 * after the sequence's last token to state_out [N, Hv, d_k, d_v].
 *   k [T,Hk,d_k], v [T,Hv,d_v] (qkv_dtype); g, beta [T,Hv] fp32.
 * workspace: device memory of at least gdn_workspace_size(..., 0) bytes,
 * 256-byte aligned; its contents on entry do not matter.
 * For bf16 inputs whose longest tail has at least 20 chunks and whose batch
 * is small enough (N x Hv x (d_v / 32 + (d_v + d_k) / 64) workgroups fit on
 * the device at once), the chain is evaluated in two halves: the state is
 * linear in the first half's state, so it is formed as the second half's
 * transition applied to the first half's state plus the second half's state
 * from zero.  The result equals the one-chain evaluation up to rounding order
 * (about 1e-6 relative); below those sizes it is the one-chain evaluation.
 */
gdn_status gdn_tail_replay(const gdn_shape* shape,
                           const int32_t* cu_seqlens_host,
                           const int32_t* cu_seqlens,
                           const void* k, const void* v,
                           const float* g, const float* beta,
                           float* state_out,
                           void* workspace, size_t workspace_bytes,
                           void* stream);

/*
 * Chunked forward over new tokens (the suffix after a rebuilt state, paper
 * Section 3): start each (sequence, value head) from state_in (NULL = zero
 * state), apply Eq. 1 to every token, write o_t = scale * S_t q_t to
 * o [T, Hv, d_v] (qkv_dtype) and, unless state_out is NULL, the final state
 * to state_out [N, Hv, d_k, d_v] (may equal state_in).
 * workspace: at least gdn_workspace_size(..., 1) bytes, 256-byte aligned.
 */
gdn_status gdn_chunk_forward(const gdn_shape* shape,
                             const int32_t* cu_seqlens_host,
                             const int32_t* cu_seqlens,
                             const void* q, const void* k, const void* v,
                             const float* g, const float* beta,
                             const float* state_in,
                             void* o, float* state_out,
                             void* workspace, size_t workspace_bytes,
                             void* stream);

/*
 * Profiling variants: identical work and results, plus stage timing.  The
 * library enqueues its kernels in gdn_num_stages(with_outputs) stages; before
 * stage i it records stage_events[i] (a hipEvent_t created by the caller) on
 * `stream`, and after the last stage it records stage_events[num_stages].
 * num_events must be gdn_num_stages(...) + 1.  Stages that have nothing to do
 * still record their event, so every event is recorded on every call.
 */
gdn_status gdn_tail_replay_profiled(const gdn_shape* shape,
                                    const int32_t* cu_seqlens_host,
                                    const int32_t* cu_seqlens,
                                    const void* k, const void* v,
                                    const float* g, const float* beta,
                                    float* state_out,
                                    void* workspace, size_t workspace_bytes,
                                    void* stream,
                                    void* const* stage_events, int32_t num_events);

gdn_status gdn_chunk_forward_profiled(const gdn_shape* shape,
                                      const int32_t* cu_seqlens_host,
                                      const int32_t* cu_seqlens,
                                      const void* q, const void* k, const void* v,
                                      const float* g, const float* beta,
                                      const float* state_in,
                                      void* o, float* state_out,
                                      void* workspace, size_t workspace_bytes,
                                      void* stream,
                                      void* const* stage_events, int32_t num_events);

/* Number of kernel stages a call enqueues, and the name of stage i:
 * tail replay (with_outputs = 0) "intra", "scan", "combine" (the last is empty
 * unless the chain runs in two halves); forward "intra", "scan". */
int32_t gdn_num_stages(int32_t with_outputs);
const char* gdn_stage_name(int32_t with_outputs, int32_t stage);

/*
 * Replay, then continue (paper Section 3: the rebuilt state S_m is the start
 * of the new suffix's prefill, Eq. 2 followed by Eq. 1 from i = m + 1).  One
 * call does what gdn_tail_replay followed by gdn_chunk_forward(state_in =
 * state_mid) does, but overlaps work that does not depend on the rebuilt
 * state: the suffix's per-chunk preparation runs beside the tail's sequential
 * scan.  The tail runs in two halves exactly where gdn_tail_replay would, so
 * the results are bit for bit those of the two calls.  Stages (for
 * gdn_replay_forward_profiled): "tail intra", "tail scan (+ suffix intra)",
 * "combine (+ suffix intra)", "suffix scan": the suffix's chunk preparation
 * runs beside the tail scan when the tail is one chain, beside the combine of
 * its two halves otherwise (the combine stage is empty for one chain).
 *   tail   (sequence n = the last r_n matched tokens, packed by cu_tail):
 *          k_tail [Tt,Hk,d_k], v_tail [Tt,Hv,d_v], g_tail, beta_tail [Tt,Hv];
 *   suffix (the new tokens of sequence n, packed by cu_suf, same N):
 *          q, k [Ts,Hk,d_k], v [Ts,Hv,d_v], g, beta [Ts,Hv];
 *   state_mid [N,Hv,d_k,d_v]: receives S_m, the replayed state (required);
 *   o [Ts,Hv,d_v]: suffix outputs; state_out: final state (NULL = not
 *   written; may equal state_mid, must not otherwise overlap it).
 * workspace: at least gdn_replay_forward_workspace_size(...) bytes, 256-byte
 * aligned.  Validation and errors as for the two separate calls.
 */
gdn_status gdn_replay_forward_workspace_size(const gdn_shape* shape,
                                             const int32_t* cu_tail_host,
                                             const int32_t* cu_suf_host,
                                             size_t* bytes);

gdn_status gdn_replay_forward(const gdn_shape* shape,
                              const int32_t* cu_tail_host, const int32_t* cu_tail,
                              const void* k_tail, const void* v_tail,
                              const float* g_tail, const float* beta_tail,
                              const int32_t* cu_suf_host, const int32_t* cu_suf,
                              const void* q, const void* k, const void* v,
                              const float* g, const float* beta,
                              float* state_mid, void* o, float* state_out,
                              void* workspace, size_t workspace_bytes,
                              void* stream);

/* Profiling variant of gdn_replay_forward, events as for the other calls;
 * num_events must be gdn_replay_forward_num_stages() + 1. */
gdn_status gdn_replay_forward_profiled(const gdn_shape* shape,
                                       const int32_t* cu_tail_host, const int32_t* cu_tail,
                                       const void* k_tail, const void* v_tail,
                                       const float* g_tail, const float* beta_tail,
                                       const int32_t* cu_suf_host, const int32_t* cu_suf,
                                       const void* q, const void* k, const void* v,
                                       const float* g, const float* beta,
                                       float* state_mid, void* o, float* state_out,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream,
                                       void* const* stage_events, int32_t num_events);

int32_t gdn_replay_forward_num_stages(void);
const char* gdn_replay_forward_stage_name(int32_t stage);

/*
 * One decode step (paper Section 2, Eq. 1 applied to a single new token; the
 * tokens generated after the prefix state has been rebuilt, Section 3).  For
 * each sequence n (num_seqs = N, one token each) and value head h, with
 * alpha = exp(g):
 *     M1 = alpha M + k (beta (v - alpha M^T k))^T,   o = scale M1^T q.
 *   q, k [N,Hk,d_k], v [N,Hv,d_v] (qkv_dtype); g, beta [N,Hv] fp32;
 *   state_in [N,Hv,d_k,d_v] fp32 (NULL = zero state); state_out (required;
 *   may equal state_in, must not otherwise overlap it); o [N,Hv,d_v].
 * No workspace; one kernel on `stream`.  q, k, v, o and the states must be
 * 16-byte aligned (GDN_ERR_UNSUPPORTED otherwise); N = 0 does nothing.
 */
gdn_status gdn_decode_step(const gdn_shape* shape,
                           const void* q, const void* k, const void* v,
                           const float* g, const float* beta,
                           const float* state_in, void* o, float* state_out,
                           void* stream);

/*
 * Tail replay that allocates nothing, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc).  Same operation, arguments, layouts and results as
 * gdn_tail_replay (the same kernels, so the states are bit for bit equal),
 * but the workspace is a device array inside the library of
 * GDN_NOALLOC_SCRATCH_BYTES bytes, one copy per GPU, held until the process
 * ends; the caller still owns k, v, g, beta and state_out.  Inputs whose
 * workspace (gdn_workspace_size(..., 0, ...)) exceeds the array are rejected
 * with GDN_ERR_WORKSPACE before anything is enqueued.  The array's device
 * address is looked up on the first call on each device (the current device
 * at the call); no call allocates, frees or synchronises.  Every call on one
 * GPU shares that GPU's array: calls that may overlap on one GPU (on
 * different streams, or from several threads without ordering) race and give
 * wrong results; order them on one stream.
 */
#define GDN_NOALLOC_SCRATCH_BYTES (64u << 20)
gdn_status gdn_tail_replay_noalloc(const gdn_shape* shape,
                                   const int32_t* cu_seqlens_host,
                                   const int32_t* cu_seqlens,
                                   const void* k, const void* v,
                                   const float* g, const float* beta,
                                   float* state_out,
                                   void* stream);

/* GDN_NOALLOC_SCRATCH_BYTES, as the library was built. */
size_t gdn_noalloc_scratch_bytes(void);

/*
 * Replay budget of the paper (Section 3): k = ceil(r * m) for a ratio
 * r = ratio_num / ratio_den, in exact integer arithmetic.  Returns -1 when
 * m < 0, ratio_num < 0, ratio_den <= 0 or the product overflows.
 */
int64_t gdn_replay_len(int64_t m, int64_t ratio_num, int64_t ratio_den);

/* Static description of a status code. */
const char* gdn_status_string(gdn_status status);

/* Detail of the last failed call on this thread ("" if none). */
const char* gdn_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GDN_TAIL_REPLAY_H */
