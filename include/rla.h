/*
 * rla.h -- C ABI of the MI355X (gfx950) library for the Residual Linear
 * Attention (RLA) and Residual Delta Net (RDN) sequence-mixing operators of
 * "Enhancing linear attention with residual learning" (Sec. 3.4, "Final
 * Formulations").
 *
 * Per sequence and head, with the paper's states S, R in R^{d_v x d_k}:
 *   x_t = v_t - S_{t-1} k_t ;  r_t = Clip_[-c,c](x_t)          (Sec. 3.1, 3.3)
 *   RDN: R_t = aR_t R_{t-1} (I - g_t k_t k_t^T) + g_t r_t k_t^T
 *        S_t = aS_t S_{t-1} (I - b_t k_t k_t^T) + b_t v_t k_t^T
 *   RLA: R_t = aR_t R_{t-1} + g_t r_t k_t^T ;  S_t = aS_t S_{t-1} + b_t v_t k_t^T
 *   o_t = aS_t S_{t-1} q_t + g_t R_t q_t
 * aS, aR are the decays of S and R (the paper ties them: pass the same
 * array twice), b = beta the write strength of S (Sec. 3.2), g = gamma the
 * correction factor (Sec. 3.2).  q and k are taken as given; the paper
 * L2-normalises them (Sec. 3.3) before the operator.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * Memory.  Every tensor pointer is DEVICE memory owned by the caller.  The
 *   library allocates nothing and keeps no state between calls; scratch
 *   space is the caller's `workspace` of at least rla_workspace_size() bytes
 *   (256-byte aligned).  Inputs are read only; outputs are fully overwritten.
 *   Calls are asynchronous on `stream` (a hipStream_t; NULL = null stream).
 * Layout (row-major, contiguous):
 *   q, k                [B, T, H, d_k]      (element type: problem.dtype)
 *   v, dO               [B, T, H, d_v]      (element type: problem.dtype)
 *   dq, dk              [B, T, H, d_k]      (element type: problem.out_dtype)
 *   o, dv               [B, T, H, d_v]      (element type: problem.out_dtype)
 *   gates and their gradients  [B, T, H]    fp32
 *   states S0, R0, S_final, R_final, dS_final, dR_final, dS0, dR0
 *                       [N, H, d_k, d_v]    fp32, where element (i, j) is the
 *                       paper's S[j][i] (the state is stored transposed)
 *   With cu_seqlens (B must be 1) the T tokens are a packing of N sequences:
 *   sequence n is tokens [cu_seqlens[n], cu_seqlens[n+1]); states reset at
 *   every sequence start.  Without it N = B sequences of length T.
 *   q, k, v, o, dO, dq, dk, dv must be 16-byte aligned.
 * Gates.  Gate values, not logits (unless RLA_FLAG_GATE_PREACT): aS, aR in
 *   (0, 1], b, g in [0, 1] are preconditions not checked on the device.
 *   Decays below 2^-126 are treated as 2^-126.
 * Clip.  clip >= 0; +INFINITY disables clipping.  The clip's derivative is
 *   taken as 1 on the closed interval [-clip, clip].
 * Errors.  Argument, shape and workspace errors are detected on the host
 *   before any HIP call and returned as a status; nothing is launched.
 *   cu_seqlens is device memory and is not read by the host: on the device
 *   sequence n spans [m_n, m_{n+1}) where m_i is the running maximum of the
 *   offsets cu[0..i] clamped into [0, T]; for increasing offsets this is
 *   [cu[n], cu[n+1]), and any other input yields disjoint, possibly empty,
 *   sequences.  Tokens outside every sequence get zero outputs/gradients.
 *   Launch failures return RLA_ERR_HIP.  No call aborts or throws.
 * Supported shapes.  bf16: d_k, d_v in {64, 128}.  fp32: d_k = 64,
 *   d_v in {64, 128} for the chunked forward (the decoding step below takes
 *   d_k in {64, 128}); the backward (and a forward with
 *   RLA_FLAG_SAVE_FOR_BACKWARD) in fp32 needs d_v = 64 and returns
 *   RLA_ERR_UNSUPPORTED otherwise.  Any B, T >= 0, H >= 1.  Internally the sequence is
 *   processed in chunks of 64 tokens; results do not depend on B or packing.
 * Precision.  fp32 inputs: fp32 arithmetic throughout.  bf16 inputs: matrix
 *   products on MFMA with fp32 accumulation; products of q or k with a state
 *   use the state split into two bf16 terms (about 16 mantissa bits, fp32
 *   range), except the backward's k dS and k dR, which use one fp16 copy of
 *   each gradient state scaled by a power of two per chunk; all other
 *   product operands are fp16 (intermediates bounded by the inputs, the clip
 *   and the gates), so bf16 q and k are expected within fp16's range, as
 *   L2-normalised rows are.  States are carried in fp32.
 *   out_dtype may be fp32 (no output rounding) or bf16 (for bf16 inputs).
 *   Backward, bf16 inputs: for each (sequence, head) the upstream gradients
 *   dO, dS_final, dR_final are multiplied by one power of two that brings
 *   their largest magnitude into [4, 8) and every gradient is multiplied back
 *   when written (exact), so any loss scale is handled alike; fp16 operands
 *   then resolve values down to about 2^-16 of that largest magnitude.
 */
#ifndef RLA_MI355X_RLA_H
#define RLA_MI355X_RLA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  RLA_OK = 0,
  RLA_ERR_NULL_ARG = 1,    /* a required pointer is NULL */
  RLA_ERR_SHAPE = 2,       /* a size is negative, inconsistent or unsupported */
  RLA_ERR_DTYPE = 3,       /* unknown dtype, or dtype not supported for the shape */
  RLA_ERR_UNSUPPORTED = 4, /* valid request this build does not implement */
  RLA_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than required */
  RLA_ERR_VALUE = 6,       /* bad scalar (clip < 0 or NaN) or misaligned pointer */
  RLA_ERR_HIP = 7,         /* a HIP runtime call or kernel launch failed */
  RLA_ERR_SCRATCH = 8      /* rdn_forward_noalloc: the problem needs more workspace
                              than RLA_NOALLOC_SCRATCH_BYTES */
} rla_status;

typedef enum { RLA_F32 = 0, RLA_BF16 = 1 } rla_dtype;

/* Operation codes for rla_workspace_size. */
typedef enum {
  RLA_OP_RLA_FORWARD = 0,
  RLA_OP_RDN_FORWARD = 1,
  RLA_OP_RDN_BACKWARD = 2,
  RLA_OP_RLA_BACKWARD = 3
} rla_op;

typedef struct {
  int64_t batch;            /* B (must be 1 when cu_seqlens != NULL) */
  int64_t seq_len;          /* T: tokens per batch row (total tokens with cu_seqlens) */
  int64_t num_heads;        /* H */
  int64_t head_dim_k;       /* d_k (= d_q) */
  int64_t head_dim_v;       /* d_v */
  int64_t num_seqs;         /* N when cu_seqlens != NULL, else ignored (N = B) */
  const int32_t *cu_seqlens;/* device pointer to N+1 offsets, or NULL */
  int32_t dtype;            /* rla_dtype of q, k, v, dO */
  float clip;               /* c >= 0, or +INFINITY for no clipping */
  int32_t out_dtype;        /* rla_dtype of o, dq, dk, dv (fp32 inputs: fp32 only) */
  uint32_t flags;           /* RLA_FLAG_* bits, 0 by default */
  const float *decay_param; /* device [2][H]: a (> 0) then b, read with RLA_FLAG_GATE_PREACT */
  float *decay_param_grad;  /* device [2][H]: d/da then d/db, written by a backward with
                               RLA_FLAG_GATE_PREACT (may be NULL: not written) */
} rla_problem;

/*
 * Save-for-backward (training).  With RLA_FLAG_SAVE_FOR_BACKWARD a forward
 * call needs a workspace of rla_workspace_size(problem, <backward op>) bytes
 * and leaves in it what the matching backward recomputes otherwise (the chunk
 * tables and matrices, the chunk-start states and the clip masks).  With
 * RLA_FLAG_USE_SAVED a backward call skips that recomputation and reads the
 * workspace instead: the caller guarantees that the last forward written to
 * that workspace had the same problem and inputs and the save flag (this
 * cannot be checked).  Without the flags every call is self-contained.
 */
#define RLA_FLAG_SAVE_FOR_BACKWARD 1u
#define RLA_FLAG_USE_SAVED 2u

/*
 * Variants of the operator (flags, any combination; every entry point
 * supports them, forward, backward and decoding alike):
 *   RLA_FLAG_RESIDUAL_TANH    r_t = c tanh(x_t / c): the negative gradient of
 *       the log-cosh loss c^2 log cosh((v - v_hat) / c), the robust
 *       alternative to the clip of App. B (c = 1 is the paper's plain tanh;
 *       c = +INFINITY gives r = x, c = 0 gives r = 0).
 *   RLA_FLAG_UNGATED_OUTPUT   o_t = S_{t-1} q_t + R_t q_t, the ungated output
 *       combination of the ablation in Sec. 4.3.
 *   RLA_FLAG_DECAYED_RESIDUAL x_t = v_t - aS_t S_{t-1} k_t, the residual of
 *       the decayed prediction (the gated rows of Table 1) instead of the
 *       boxed v_t - S_{t-1} k_t.
 * A backward with RLA_FLAG_USE_SAVED must carry the variant flags of the
 * saving forward.
 */
#define RLA_FLAG_RESIDUAL_TANH 4u
#define RLA_FLAG_UNGATED_OUTPUT 8u
#define RLA_FLAG_DECAYED_RESIDUAL 16u

/*
 * Input pre-processing inside the operator (the closing paragraph of
 * Sec. 3.4 and the caption of the architecture figure; any combination, every
 * entry point; gradients are with respect to the raw inputs):
 *   RLA_FLAG_QK_SILU_L2NORM  q and k are raw projections: each token-head row
 *       becomes y / max(||y||, 1e-12) with y = SiLU(x) before the recurrence
 *       (the torch F.normalize convention).  bf16 inputs: the normalised rows
 *       are rounded to bf16 once.  Needs workspace (rla_workspace_size).
 *   RLA_FLAG_GATE_PREACT  alpha_s, alpha_r, beta, gamma hold pre-activations z:
 *       aS = exp(-a_h softplus(z + b_h)) (likewise aR, with the same per-head
 *       (a_h, b_h) from problem.decay_param: the Mamba-2 re-parameterisation),
 *       beta = sigmoid(z), gamma = sigmoid(z).  The backward returns the
 *       gradients of the pre-activations and, in problem.decay_param_grad,
 *       of (a_h, b_h) summed over every token and both decays.
 */
#define RLA_FLAG_QK_SILU_L2NORM 32u
#define RLA_FLAG_GATE_PREACT 64u

/* Bytes of workspace the operation needs for this problem (0 if the problem
 * is invalid).  Pure host function. */
size_t rla_workspace_size(const rla_problem *problem, int op);

/*
 * Profiling aid (opt-in, per calling thread): while `events` is non-NULL,
 * each later forward/backward call on this thread records events[0] on its
 * stream when its first kernel stage starts and events[i] after stage i,
 * up to num_events events.  Stages: forward = {prep, scan}; backward =
 * {prep, checkpointing forward scan (these two are skipped with
 * RLA_FLAG_USE_SAVED), upstream-gradient maxima (bf16 inputs only), reverse
 * scan, gradient kernel}.
 * The events are hipEvent_t handles owned by the caller.  NULL turns it off.
 */
void rla_set_stage_events(void **events, int num_events);

/* Human-readable name of a status code (static string). */
const char *rla_status_string(rla_status status);

/*
 * RLA forward (paper Sec. 3.4, left box): additive base state S and additive
 * residual state R.  S0/R0 may be NULL (zero initial states); S_final/R_final
 * may be NULL (not written).  o is [B, T, H, d_v] in problem.out_dtype.
 */
rla_status rla_forward(const rla_problem *problem,
                       const void *q, const void *k, const void *v,
                       const float *alpha_s, const float *beta,
                       const float *alpha_r, const float *gamma,
                       const float *S0, const float *R0,
                       void *o, float *S_final, float *R_final,
                       void *workspace, size_t workspace_bytes, void *stream);

/*
 * RDN forward (paper Sec. 3.4, right box): gated delta-rule base state S and
 * gated delta-rule residual state R.  Arguments as for rla_forward.
 */
rla_status rdn_forward(const rla_problem *problem,
                       const void *q, const void *k, const void *v,
                       const float *alpha_s, const float *beta,
                       const float *alpha_r, const float *gamma,
                       const float *S0, const float *R0,
                       void *o, float *S_final, float *R_final,
                       void *workspace, size_t workspace_bytes, void *stream);

/*
 * Allocation-free RDN forward, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): rdn_forward with the workspace taken from a static device array
 * of RLA_NOALLOC_SCRATCH_BYTES (128 MiB) inside the library instead of an
 * argument.  Each GPU the library runs on holds its own array from the first
 * call on it until the process ends; the call uses the array of the calling
 * thread's current device, so `stream` must belong to that device.  The call
 * allocates nothing and launches only the kernels rdn_forward launches (no
 * memset nodes).  Problems whose rla_workspace_size(problem,
 * RLA_OP_RDN_FORWARD) exceeds the array return RLA_ERR_SCRATCH before any HIP
 * call (bf16, H = 16, d = 128, one sequence: up to 19,648 tokens);
 * RLA_FLAG_SAVE_FOR_BACKWARD and RLA_FLAG_USE_SAVED are rejected
 * (RLA_ERR_VALUE).  The array keeps the last call's contents; nothing in it
 * needs to start at zero.  All calls on one GPU share its array: calls that
 * overlap in time on one GPU (other streams, other threads) race and must be
 * serialised by the caller.  Other arguments and results as rdn_forward.
 */
#define RLA_NOALLOC_SCRATCH_BYTES (128u << 20)
rla_status rdn_forward_noalloc(const rla_problem *problem,
                               const void *q, const void *k, const void *v,
                               const float *alpha_s, const float *beta,
                               const float *alpha_r, const float *gamma,
                               const float *S0, const float *R0,
                               void *o, float *S_final, float *R_final, void *stream);

/*
 * RDN backward: gradients of L = <dO, o> + <dS_final, S_T> + <dR_final, R_T>
 * with respect to every input of rdn_forward.  By default the call recomputes
 * the forward from the inputs; with RLA_FLAG_USE_SAVED it reads what a
 * forward with RLA_FLAG_SAVE_FOR_BACKWARD left in the same workspace instead
 * (see the save-for-backward flags above).  dS_final, dR_final, S0, R0 may be
 * NULL (zeros); dS0, dR0 may be NULL (not written).  dq, dk, dv are in
 * problem.out_dtype; gate gradients are fp32 and are with respect to the
 * gate values (not their logarithms).
 */
rla_status rdn_backward(const rla_problem *problem,
                        const void *q, const void *k, const void *v,
                        const float *alpha_s, const float *beta,
                        const float *alpha_r, const float *gamma,
                        const float *S0, const float *R0,
                        const void *dO, const float *dS_final, const float *dR_final,
                        void *dq, void *dk, void *dv,
                        float *dalpha_s, float *dbeta, float *dalpha_r, float *dgamma,
                        float *dS0, float *dR0,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * RLA backward: as rdn_backward, for rla_forward (paper Sec. 3.4, left box).
 */
rla_status rla_backward(const rla_problem *problem,
                        const void *q, const void *k, const void *v,
                        const float *alpha_s, const float *beta,
                        const float *alpha_r, const float *gamma,
                        const float *S0, const float *R0,
                        const void *dO, const float *dS_final, const float *dR_final,
                        void *dq, void *dk, void *dv,
                        float *dalpha_s, float *dbeta, float *dalpha_r, float *dgamma,
                        float *dS0, float *dR0,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * Recurrent step for decoding (the token recurrence of Sec. 3.4 evaluated
 * directly, as in the paper's recurrent pseudo-code of App. D): advances the
 * states of B = problem.batch sequences by T = problem.seq_len tokens each
 * and writes the T outputs.  Meant for small T (T = 1 per generated token);
 * the chunked rla_forward / rdn_forward serve long sequences.
 *   q, k [B, T, H, d_k], v [B, T, H, d_v]      problem.dtype
 *   alpha_s, beta, alpha_r, gamma [B, T, H]     fp32 gate values
 *   o [B, T, H, d_v]                            problem.out_dtype
 *   S_in, R_in [B, H, d_k, d_v] fp32, or NULL for zero states
 *   S_out, R_out [B, H, d_k, d_v] fp32, required, 16-byte aligned; S_out may
 *     be the same pointer as S_in (in-place update), likewise R_out and R_in;
 *     any other overlap among the four state buffers is rejected.
 * No workspace.  problem.cu_seqlens must be NULL (RLA_ERR_UNSUPPORTED).
 * problem.flags may carry the variant flags (RLA_FLAG_RESIDUAL_TANH,
 * RLA_FLAG_UNGATED_OUTPUT, RLA_FLAG_DECAYED_RESIDUAL) and the pre-processing
 * flags (RLA_FLAG_QK_SILU_L2NORM, RLA_FLAG_GATE_PREACT), applied to each
 * token as in the chunked entry points; RLA_FLAG_SAVE_FOR_BACKWARD and
 * RLA_FLAG_USE_SAVED are rejected (RLA_ERR_VALUE).
 * bf16 and fp32 inputs both support d_k, d_v in {64, 128};
 * all arithmetic is fp32 (bf16 inputs are widened exactly).  Decays are used
 * as given (no 2^-126 floor is needed here).  T = 0 copies S_in, R_in (or
 * zeros) to S_out, R_out.  Each (sequence, head) reads its states once and
 * writes them once, so a step moves 16 d_k d_v bytes per (sequence, head).
 */
rla_status rla_decode(const rla_problem *problem,
                      const void *q, const void *k, const void *v,
                      const float *alpha_s, const float *beta,
                      const float *alpha_r, const float *gamma,
                      const float *S_in, const float *R_in,
                      void *o, float *S_out, float *R_out, void *stream);

/* RDN recurrent step (Sec. 3.4, right box); arguments as for rla_decode. */
rla_status rdn_decode(const rla_problem *problem,
                      const void *q, const void *k, const void *v,
                      const float *alpha_s, const float *beta,
                      const float *alpha_r, const float *gamma,
                      const float *S_in, const float *R_in,
                      void *o, float *S_out, float *R_out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* RLA_MI355X_RLA_H */
