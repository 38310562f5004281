/*
 * gdr2.h -- C ABI of the MI355X (gfx950) chunkwise Gated Delta Rule-2 operator.
 *
 * Gated Delta Rule-2 (Gated DeltaNet-2, arXiv 2605.22791, Sec. 3.1, eqs.
 * eq_gdn2_e_z, eq_gdn2_residual, eq_gdn2_recurrence).  For every batch row b
 * and head h independently, with state S in R^{Dk x Dv}:
 *
 *     e_t = b_t * k_t,   z_t = w_t * v_t                 (erase / write factors)
 *     S_t = (I - k_t e_t^T) Diag(exp(g_t)) S_{t-1} + k_t z_t^T
 *     o_t = scale * S_t^T q_t                            (post-update read-out)
 *
 * g = log_alpha is the per-key-channel log-decay (the paper's g_t; alpha_t =
 * exp(g_t)), b in [0,1]^Dk (or [0,2]^Dk for the negative-eigenvalue variant,
 * Sec. 3.1) is the erase gate and w in [0,1]^Dv the write gate.  `scale`
 * multiplies the output only (callers normally pass 1/sqrt(Dk); the paper's
 * notation is scale = 1).  q and k are consumed as given: L2 normalisation,
 * when wanted (App. D.2), is the caller's.
 *
 * T need not be a multiple of the chunk length: the last chunk of every
 * sequence may be partial.
 *
 * Layout and dtypes (all tensors contiguous, row-major, device memory; Hv =
 * H unless grouped value heads are asked for, see gdr2_problem):
 *     q, k, b, log_alpha           (B, T, H, Dk)
 *     v, w, o                      (B, T, Hv, Dv)
 *     S0, S_T, S, dS_T, dS0        (B, Hv, Dk, Dv)  always fp32
 *     log_alpha, dlog_alpha        always fp32 (the decay is formed in fp32,
 *                                  App. C.1 / App. D.1)
 *     q, k, v, b, w, o, dout, dq, dk, dv, db, dw
 *                                  problem->dtype (bf16 or fp32)
 * The recurrent state is fp32 everywhere (App. D.3); every product inside the
 * kernels accumulates in fp32.
 *
 * Ownership and errors:
 *   * The caller owns every buffer; the library never allocates device memory
 *     and keeps no mutable global state (apart from the opt-in, per-thread
 *     kernel timing at the end of this header, and the fixed per-GPU array of
 *     gdr2_chunk_fwd_noalloc), so calls are re-entrant (gdr2_chunk_fwd_noalloc:
 *     see its own rules).
 *     Work is enqueued on `stream` and the call returns without waiting.
 *   * Outputs are overwritten, never accumulated.  Workspace contents are
 *     undefined after a call.  Inputs and outputs must not alias (except S in
 *     gdr2_recurrent_step, which is updated in place).
 *   * Every argument is validated before any HIP call; on error nothing is
 *     launched and the status says why:
 *       GDR2_EINVAL        null required pointer, pointer not 16-byte aligned
 *                          (cu_seqlens: 4-byte aligned), a dimension <= 0,
 *                          non-finite scale, unknown dtype, Hv not a
 *                          multiple of H, n_seqs <= 0 or B != 1 in a
 *                          packed call;
 *       GDR2_EUNSUPPORTED  Dk or Dv not in {64, 128}, chunk != 64, sizes
 *                          beyond 2^31 elements per tensor, more than 2^24
 *                          sequences in a packed call;
 *       GDR2_EWORKSPACE    ws_bytes below gdr2_chunk_workspace_bytes();
 *       GDR2_EHIP          a launch reported an error (hipGetLastError).
 *   * No C++ exception crosses this interface.
 *   * Setting the environment variable GDR2_DEBUG_SYNC=1 (read once, at the
 *     first call) makes every call wait for its stream after its launches and
 *     report an asynchronous kernel failure as GDR2_EHIP; it changes no result
 *     and no schedule.  Nothing else in the environment is read.
 *   * Inputs outside the documented domain (log_alpha > 0, NaN/Inf values)
 *     are not checked; results are then undefined.
 */
#ifndef GDR2_H_
#define GDR2_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum gdr2_status {
  GDR2_OK = 0,
  GDR2_EINVAL = 1,
  GDR2_EUNSUPPORTED = 2,
  GDR2_EWORKSPACE = 3,
  GDR2_EHIP = 4
} gdr2_status;

typedef enum gdr2_dtype { GDR2_BF16 = 0, GDR2_FP32 = 1 } gdr2_dtype;

/* Problem description shared by every call.  `chunk` must be 64 (the chunk
 * length C of Sec. 3.3; App. C.2 fixes C = 64).  Hv: value heads (0 means
 * Hv = H); grouped value heads (Sec. 3.5, App. C.1) have Hv = G * H: value
 * head j uses key head j / G, i.e. q, k, log_alpha and b (H heads) are
 * repeated across each group of G consecutive value heads, while v, w, o,
 * dout and every state live on the Hv value heads.  dq, dk, db and
 * dlog_alpha are then the sums over the group. */
typedef struct gdr2_problem {
  int32_t B, T, H, Dk, Dv;
  int32_t chunk;
  float scale;
  int32_t dtype; /* gdr2_dtype */
  int32_t Hv;    /* value heads, a multiple of H; 0: Hv = H */
} gdr2_problem;

/* Bytes of device workspace a chunk call needs (for_backward = 0: forward,
 * 1: backward).  Writes the size to *bytes.  Errors as in the calls. */
gdr2_status gdr2_chunk_workspace_bytes(const gdr2_problem* problem, int for_backward,
                                       size_t* bytes);

/* Chunkwise WY forward (Sec. 3.3; App. A; App. C.2): the intra-chunk kernel
 * forms the decay-weighted Gram T = tril(Ebar Kbar^T, -1) and the scores A_qk,
 * solves A = (I + T)^{-1} in fp32 and builds Y = A Ebar and U = A (W*V); the
 * state kernel then carries S across chunks (eq. eq_gdn2_chunk_state) and
 * writes O (eq. eq_gdn2_chunk_output).
 *   S0   may be NULL (zero start state).
 *   o    receives (B,T,Hv,Dv) in problem->dtype.
 *   S_T  may be NULL; otherwise receives the final state (fp32).
 *   ws   device workspace of at least gdr2_chunk_workspace_bytes(p, 0). */
gdr2_status gdr2_chunk_fwd(const gdr2_problem* problem, const void* q, const void* k,
                           const void* v, const float* log_alpha, const void* b,
                           const void* w, const float* S0, void* o, float* S_T, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* Maximum workspace of gdr2_chunk_fwd_noalloc: the size of its fixed array. */
#define GDR2_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): exactly
 * gdr2_chunk_fwd, with no workspace argument.  Its workspace is one fixed
 * __device__ array of GDR2_NOALLOC_SCRATCH_BYTES (64 MiB) per GPU, which the
 * library holds on every GPU it runs on until the process ends; the call
 * itself allocates nothing and issues no memset.
 *   * Runs on the current device; `stream` must belong to it.
 *   * GDR2_EWORKSPACE: the problem needs more than GDR2_NOALLOC_SCRATCH_BYTES
 *     of workspace (gdr2_chunk_workspace_bytes(p, 0) tells), e.g. more than
 *     about 450 chunk-heads at Dk = Dv = 128; nothing is launched.
 *   * Every call on one GPU uses that GPU's array: calls that overlap on one
 *     GPU (other streams, other threads, without ordering between them) race
 *     and give undefined results.  Calls ordered on one stream are safe.
 *   * Other arguments, validation (before any HIP call) and errors as in
 *     gdr2_chunk_fwd; GDR2_EHIP also when the array's device address cannot be
 *     looked up. */
gdr2_status gdr2_chunk_fwd_noalloc(const gdr2_problem* problem, const void* q, const void* k,
                                   const void* v, const float* log_alpha, const void* b,
                                   const void* w, const float* S0, void* o, float* S_T,
                                   hipStream_t stream);

/* Gate-aware chunkwise backward (Sec. 3.4; App. B; App. C.3) of
 *     L = sum_t <o_t, dout_t> + <S_T, dS_T>
 * with respect to every input.  The forward intermediates are recomputed from
 * the inputs (the memory-saving path of App. D.3), so the call takes exactly
 * the forward's inputs plus the upstream gradients.
 *   S0, dS_T   may be NULL (zero).
 *   dq, dk, db (B,T,H,Dk) and dv, dw (B,T,Hv,Dv) in problem->dtype;
 *   dlog_alpha (B,T,H,Dk) fp32; dS0 (B,Hv,Dk,Dv) fp32 or NULL (not wanted).
 *   ws   device workspace of at least gdr2_chunk_workspace_bytes(p, 1). */
gdr2_status gdr2_chunk_bwd(const gdr2_problem* problem, const void* q, const void* k,
                           const void* v, const float* log_alpha, const void* b,
                           const void* w, const float* S0, const void* dout,
                           const float* dS_T, void* dq, void* dk, void* dv,
                           float* dlog_alpha, void* db, void* dw, float* dS0, void* ws,
                           size_t ws_bytes, hipStream_t stream);

/* Training path that keeps the forward's intermediates instead of recomputing
 * them (App. D.3 names recomputation as the memory-saving path; a8 of the
 * backward then reads h_n, R and A as stored).  gdr2_chunk_fwd_save computes
 * exactly what gdr2_chunk_fwd computes and additionally leaves in ws the
 * intra-chunk tiles, A = (I + T)^{-1}, the chunk-start states h_n and R_n;
 * gdr2_chunk_bwd_saved returns exactly what gdr2_chunk_bwd returns but reads
 * those instead of recomputing them (it skips the two recompute kernels).
 *   * ws must hold at least gdr2_chunk_workspace_bytes(p, 1) bytes for both
 *     calls, and must not be written between them.
 *   * The two calls must get the same problem, q, k, v, log_alpha, b, w and
 *     S0 (the saved states already contain S0); otherwise the gradients are
 *     undefined.  Other arguments, errors and ownership as in gdr2_chunk_fwd /
 *     gdr2_chunk_bwd. */
gdr2_status gdr2_chunk_fwd_save(const gdr2_problem* problem, const void* q, const void* k,
                                const void* v, const float* log_alpha, const void* b,
                                const void* w, const float* S0, void* o, float* S_T, void* ws,
                                size_t ws_bytes, hipStream_t stream);
gdr2_status gdr2_chunk_bwd_saved(const gdr2_problem* problem, const void* q, const void* k,
                                 const void* v, const float* log_alpha, const void* b,
                                 const void* w, const float* S0, const void* dout,
                                 const float* dS_T, void* dq, void* dk, void* dv,
                                 float* dlog_alpha, void* db, void* dw, float* dS0, void* ws,
                                 size_t ws_bytes, hipStream_t stream);

/* Recurrent (token-by-token) forward for decoding (App. C.5): applies the
 * update to problem->T >= 1 consecutive tokens (T = 1 for one decode step),
 * keeping S in fp32 and updating it in place; o (B,T,H,Dv) in problem->dtype.
 * `chunk` is ignored and T need not be a multiple of 64.  No workspace. */
gdr2_status gdr2_recurrent_step(const gdr2_problem* problem, const void* q, const void* k,
                                const void* v, const float* log_alpha, const void* b,
                                const void* w, float* S, void* o, hipStream_t stream);

/* ---- packed variable-length sequences (App. C.6) -------------------------
 * A packed batch holds n_seqs sequences end to end along T: problem->B must be
 * 1, problem->T is the total token count, and sequence s owns tokens
 * cu_seqlens[s] .. cu_seqlens[s+1) of q, k, v, log_alpha, b, w, o, dout and
 * of every token gradient.  cu_seqlens is a device array of n_seqs + 1 int32
 * offsets with 0 = cu[0] <= cu[1] <= ... <= cu[n_seqs] = T (empty sequences
 * allowed).  Each sequence is chunked on its own (its last chunk may be
 * partial), so the state restarts at every sequence boundary: the result for
 * sequence s equals a separate call on its tokens alone.  The states S0, S_T,
 * dS_T, dS0 and S (recurrent) are (n_seqs, Hv, Dk, Dv) fp32.
 * The offsets are read on the device and not checked on the host: the
 * kernels clamp them into [0, T], so malformed offsets cannot cause accesses
 * outside the tensors or the workspace, but the results are then undefined.
 * Errors, ownership and streams as for the fixed-length calls. */

/* Workspace bytes of a packed chunk call (for_backward as in
 * gdr2_chunk_workspace_bytes). */
gdr2_status gdr2_varlen_workspace_bytes(const gdr2_problem* problem, int32_t n_seqs, int for_backward,
                                        size_t* bytes);

/* Chunk forward of a packed batch.  save = 0 is gdr2_chunk_fwd (workspace of
 * gdr2_varlen_workspace_bytes(p, n, 0)), save = 1 is gdr2_chunk_fwd_save
 * (workspace of gdr2_varlen_workspace_bytes(p, n, 1)). */
gdr2_status gdr2_chunk_fwd_varlen(const gdr2_problem* problem, const int32_t* cu_seqlens, int32_t n_seqs,
                                  const void* q, const void* k, const void* v, const float* log_alpha,
                                  const void* b, const void* w, const float* S0, void* o, float* S_T,
                                  void* ws, size_t ws_bytes, int save, hipStream_t stream);

/* Chunk backward of a packed batch.  saved = 0 recomputes the forward's
 * intermediates (gdr2_chunk_bwd), saved = 1 reads those a save = 1 forward
 * left in ws (gdr2_chunk_bwd_saved; same problem, cu_seqlens and inputs). */
gdr2_status gdr2_chunk_bwd_varlen(const gdr2_problem* problem, const int32_t* cu_seqlens, int32_t n_seqs,
                                  const void* q, const void* k, const void* v, const float* log_alpha,
                                  const void* b, const void* w, const float* S0, const void* dout,
                                  const float* dS_T, void* dq, void* dk, void* dv, float* dlog_alpha,
                                  void* db, void* dw, float* dS0, void* ws, size_t ws_bytes, int saved,
                                  hipStream_t stream);

/* Recurrent forward of a packed batch (App. C.5 / C.6): every sequence's
 * tokens in order, its state S[s] updated in place. */
gdr2_status gdr2_recurrent_varlen(const gdr2_problem* problem, const int32_t* cu_seqlens, int32_t n_seqs,
                                  const void* q, const void* k, const void* v, const float* log_alpha,
                                  const void* b, const void* w, float* S, void* o, hipStream_t stream);

/* ---- fused input stage (App. C.1; App. D.1 - D.2) -------------------------
 * Variants of the calls above that take the layer's raw projections and do
 * the two steps between them and the recurrence inside the kernels:
 *   * q and k are L2-normalised per (token, key head) before the update
 *     (App. D.2), read here as  y = x * (sum_c x_c^2 + eps)^(-1/2)  (the paper
 *     gives no epsilon; eps = 0 is the plain x / ||x||, which is not finite for
 *     an all-zero row);
 *   * the log-decay is formed in fp32 from the decay projection f as
 *     g = -exp(a_log[h]) * softplus(f + delta[h][c])  (eq. eq_gdn2_decay_param,
 *     App. C.1): one a_log per key head, broadcast over its Dk channels, and
 *     one delta per key channel.
 * The normalised q, k and g never exist in memory.  The backward returns the
 * gradients of the raw inputs: dq, dk through the normalisation VJP
 * dx = r (dy - y <y, dy>) (r the inverse norm, y = r x), df = dg * (-exp(a)
 * sigmoid(f + delta)), da[h] = sum over tokens, value heads of the group and
 * channels of dg * g, ddelta[h][c] = sum over tokens and group of df.
 * Everything else (shapes, S0, states, grouped value heads, packed batches with
 * cu_seqlens and n_seqs > 0, or n_seqs = 0 and cu_seqlens ignored for fixed
 * length, the stored and recomputing training paths) is as in the plain calls;
 * q, k and f take the places of q, k and log_alpha with the same shapes
 * ((B,T,H,Dk); f fp32).  bf16 problems do the stage inside the chunk kernels;
 * fp32 problems (the parity mode) run it as passes of its own around the fp32
 * operator, with the normalised q, k and g in the workspace; the recurrent
 * call does it per token for both dtypes.  The workspace
 * (gdr2_fused_workspace_bytes) adds the inverse norms of q and k and the
 * gradients of the normalised q, k (saving forward and backward), the
 * decay-parameter partials (backward) and, for fp32 problems, the stage's
 * outputs; a saving forward and the backward that reads it need the same
 * stage. */
typedef struct gdr2_stage {
  const float* a_log; /* (H) fp32, device, 4-byte aligned */
  const float* delta; /* (H, Dk) fp32, device, 16-byte aligned */
  float eps;          /* finite, >= 0 */
} gdr2_stage;

/* Workspace bytes of a fused chunk call (n_seqs = 0: fixed length; for_backward
 * as in gdr2_chunk_workspace_bytes: 1 for a saving forward and the backward). */
gdr2_status gdr2_fused_workspace_bytes(const gdr2_problem* problem, int32_t n_seqs, int for_backward,
                                       size_t* bytes);

/* Chunk forward from the raw projections (save as in gdr2_chunk_fwd_varlen). */
gdr2_status gdr2_fused_fwd(const gdr2_problem* problem, const gdr2_stage* stage, const int32_t* cu_seqlens,
                           int32_t n_seqs, const void* q, const void* k, const void* v, const float* f,
                           const void* b, const void* w, const float* S0, void* o, float* S_T, void* ws,
                           size_t ws_bytes, int save, hipStream_t stream);

/* Chunk backward from the raw projections: dq, dk (B,T,H,Dk) in the dtype,
 * df (B,T,H,Dk) fp32, da (H) fp32, ddelta (H,Dk) fp32 (16-byte aligned); the
 * other gradients as in gdr2_chunk_bwd.  All outputs are overwritten. */
gdr2_status gdr2_fused_bwd(const gdr2_problem* problem, const gdr2_stage* stage, const int32_t* cu_seqlens,
                           int32_t n_seqs, const void* q, const void* k, const void* v, const float* f,
                           const void* b, const void* w, const float* S0, const void* dout, const float* dS_T,
                           void* dq, void* dk, void* dv, float* df, float* da, float* ddelta, void* db, void* dw,
                           float* dS0, void* ws, size_t ws_bytes, int saved, hipStream_t stream);

/* Recurrent forward (decoding) from the raw projections (App. C.5): as
 * gdr2_recurrent_step / gdr2_recurrent_varlen; normalisation in fp32. */
gdr2_status gdr2_fused_recurrent(const gdr2_problem* problem, const gdr2_stage* stage, const int32_t* cu_seqlens,
                                 int32_t n_seqs, const void* q, const void* k, const void* v, const float* f,
                                 const void* b, const void* w, float* S, void* o, hipStream_t stream);

/* Static, human-readable name of a status code. */
const char* gdr2_status_str(gdr2_status status);

/* ---- measurement support (not part of the operator) ----------------------
 * Kernel identifiers used by the per-kernel timing below. */
typedef enum gdr2_kernel_id {
  GDR2_K_FWD_INTRA = 0,           /* forward: intra-chunk Gram / WY solve / Y, U   */
  GDR2_K_FWD_STATE = 1,           /* forward: inter-chunk state scan + output      */
  GDR2_K_BWD_RECOMPUTE_INTRA = 2, /* backward: intra-chunk recompute              */
  GDR2_K_BWD_RECOMPUTE_STATE = 3, /* backward: chunk-state recompute              */
  GDR2_K_BWD_STATE = 4,           /* backward: reverse state scan                 */
  GDR2_K_BWD_WY = 5,              /* backward: gate-aware WY VJP (fp32 problems)  */
  GDR2_K_BWD_INTRA = 6,           /* backward: intra-chunk VJP + decay chain (bf16
                                     problems: with the WY VJP, one kernel)      */
  GDR2_K_RECURRENT = 7,           /* recurrent / decode                           */
  GDR2_K_STAGE_BWD = 8,           /* fused stage: normalisation VJP, decay-
                                     parameter sums                              */
  GDR2_K_STAGE_FWD = 9,           /* fused stage of fp32 problems: normalisation
                                     and activation pass                         */
  GDR2_NUM_KERNELS = 10
} gdr2_kernel_id;

/* Per-thread kernel timing for benchmarks: while enabled, each kernel launched
 * by the calling thread is bracketed by two hipEvents recorded on its launch
 * stream.  gdr2_profile_collect() waits for the recorded events, writes the
 * accumulated milliseconds and launch counts of every kernel id into ms[] and
 * launches[] (n >= GDR2_NUM_KERNELS entries, else GDR2_EINVAL) and resets the
 * totals.  Off by default; costs nothing when off. */
gdr2_status gdr2_profile_enable(int on);
gdr2_status gdr2_profile_collect(double* ms, long long* launches, int n);

#ifdef __cplusplus
}
#endif

#endif /* GDR2_H_ */
