/*
 * gla.h -- C ABI of the MI355X (gfx950) chunkwise gated linear attention layer.
 *
 * The layer (Yang et al., "Gated Linear Attention Transformers with
 * Hardware-Efficient Training", Sec. 4.1, Eq. 3), per batch row b and head h:
 *
 *     S_t = Diag(alpha_t) S_{t-1} + k_t^T v_t,     o_t = q_t S_t,
 *
 * with alpha_t = exp(log_alpha_t) in (0, 1]^{d_k}, S_t in R^{d_k x d_v}, and
 * S_0 = S0 (zero, or the final state of the previous segment: Sec. 2.2).  The
 * library evaluates it in the chunkwise form of Sec. 4.2 with the secondary
 * (sub-chunk) tiling of Sec. 4.3: an inter-chunk state pass, attention-like
 * intra-chunk blocks (bf16 matrix-core products between sub-chunks, with
 * normalisers at the sub-chunk boundaries; inside a sub-chunk, Eq. 4 itself
 * in fp32 on the vector ALUs: one exponential of the log-space difference
 * per pair and feature; with a scalar gate or none, every block is the
 * plain (Q K^T) (.) D, D_ij = exp(c_i - c_j), in fp32 on the matrix cores),
 * and the closed-form gate gradient of Sec. 4.3 in
 * the backward.
 *
 * Conventions shared by every entry point
 *   - Tensors are device pointers, contiguous row-major:
 *       q, k, log_alpha, dq, dk, dlog_alpha : [B, H, T, d_k]   (io dtype)
 *       v, o, dO, dv                        : [B, H, T, d_v]   (io dtype)
 *       S0, S_T, dS_T, dS0                  : [B, H, d_k, d_v] (fp32 always)
 *     and 16-byte aligned.  "Nullable" pointers may be NULL: an absent S0 or
 *     dS_T means zero, an absent S_T or dS0 means "not wanted".
 *     With GLA_FLAG_SCALAR_GATE, log_alpha and dlog_alpha are [B, H, T].
 *   - log_alpha is nullable everywhere: NULL means alpha = 1 for every t and
 *     feature, i.e. ungated linear attention (the alpha = 1 case that the
 *     paper's FLA algorithms of Sec. 3.3 and App. A compute).  No gate tensor
 *     is then read, and the backward's dlog_alpha may be NULL too.  A NULL
 *     dlog_alpha always means the gate gradient is not wanted.  With no gate
 *     the intra-chunk blocks are plain masked q k^T products and q, k are
 *     read in place of the gated operands; with no gate and no gate gradient
 *     the backward also multiplies its states as single bf16 operands (as the
 *     forward does), since no gate-gradient sum needs their extra precision.
 *   - The caller owns every buffer; the library never allocates or frees
 *     device memory and keeps no mutable global state, so calls are
 *     re-entrant.  Outputs are overwritten, never accumulated into, and must
 *     not alias inputs.
 *   - All work is enqueued on `stream` (a hipStream_t; NULL = the default
 *     stream) and the call returns without synchronising.
 *   - Argument errors are reported synchronously, before anything is
 *     enqueued.  A failed kernel launch returns GLA_ERR_HIP; faults inside
 *     kernels surface at the caller's next synchronisation.  No C++
 *     exception crosses this boundary.
 *   - Domain: log_alpha must be finite and <= 0 (alpha in (0, 1], Sec. 4.1);
 *     log_alpha = 0 (alpha = 1) gives ungated linear attention (Sec. 2.1).
 *     Steep gates are exact: every exponent the kernels evaluate is <= 0
 *     (tested with per-step log alpha down to -50).
 *   - There is no scale argument (Eq. 3 has none): pre-scale k if desired.
 *
 * Few heads, long sequences: when B*H is too small to fill the GPU and T is
 * a multiple of the chunk, the chunkwise calls split each head's sequence into
 * segments of whole chunks, run them as separate heads and join them with
 * segment scans over the chunk decays (the two-stage form of App. A.2).  This
 * is decided from the shape alone (so gla_workspace_bytes accounts for it and
 * a forward's workspace stays valid for the backward's reuse flag), changes
 * only the summation order, and keeps the stage selector's meaning (forward
 * stage 2 then holds both state passes and the scan; backward stage 1 also
 * rebuilds the segments' initial states, stage 2 also their final-state
 * gradients).  GLA_SEGMENTS(n) in the flags fixes the segment count instead,
 * up to one chunk per segment (materialized chunk states).  The general form
 * (value-side gate) is never segmented.
 *
 * Supported shapes: B*H <= 65535; d_k and d_v multiples of 16 with d_k <= 256
 * and d_v <= 1024 (fp32 io additionally needs d_k <= 128); chunk C in
 * {16, 32, 64}; sub-chunk c a divisor of 16 that also divides C; any T >= 0
 * (a last, shorter chunk is handled by masking) with at most 65535 chunks
 * (T <= 65535 C) in the chunkwise calls and T * max(d_k, d_v) < 2^29 per
 * head.  Other values return GLA_ERR_UNSUPPORTED.  The kernels tile every
 * chunk in 16-row sub-chunk blocks: a sub-chunk length c < 16 lies inside
 * those blocks, whose fp32 evaluation does not depend on c, so every c that
 * divides 16 gives the same results (bit for bit).
 */
#ifndef GLA_H_
#define GLA_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GLA_OK = 0,
  GLA_ERR_NULL = 1,        /* a required pointer is NULL                       */
  GLA_ERR_SHAPE = 2,       /* a dimension is negative or inconsistent          */
  GLA_ERR_DTYPE = 3,       /* unknown io dtype                                 */
  GLA_ERR_UNSUPPORTED = 4, /* valid, but outside what the kernels implement    */
  GLA_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than required          */
  GLA_ERR_HIP = 6,         /* a HIP runtime call or kernel launch failed       */
  GLA_ERR_SCRATCH = 7      /* gla_chunk_fwd_noalloc: the problem needs more
                            * workspace than the library's fixed scratch array */
} gla_status;

typedef enum { GLA_F32 = 0, GLA_BF16 = 1 } gla_dtype;

/* Flags (bitwise OR) for gla_problem.flags. */
enum {
  /* gla_chunk_bwd only: the workspace still holds what gla_chunk_fwd left in
   * it for exactly the same problem and inputs (the gated operands Q (.) Lambda,
   * K (.) Gamma, the intra-chunk matrices P and the chunk decays gamma), so
   * the backward skips recomputing them (paper, Sec. 3.3: materialize once
   * vs. recompute). */
  GLA_FLAG_REUSE_FWD_WORKSPACE = 1u << 0,
  /* Data-dependent scalar gates (Table 1: the Mamba-2, mLSTM and Gated
   * Retention rows, G_t = gamma_t 1^T 1): log_alpha holds one log gamma per
   * step and head, [B, H, T] (io dtype), shared by every key feature, i.e.
   * alpha_t = gamma_t 1; the backward's dlog_alpha is then [B, H, T] too, the
   * sum over the key features of the per-feature gate gradient (summed in a
   * fixed order: reproducible bits).  Combines with gate_tau (z then [B, H, T]:
   * gamma = sigmoid(z)^(1/tau), Gated Retention; tau = 1, mLSTM).  Every entry
   * point honours it, gla_workspace_bytes included (the backward then needs
   * B H ceil(d_k/32) T fp32 more). */
  GLA_FLAG_SCALAR_GATE = 1u << 1,
  /* Accepted for compatibility and without effect: every diagonal (within
   * one sub-chunk) block of the intra-chunk terms, forward and backward, is
   * always evaluated in fp32 log space, one exponential exp(B_i - B_j) per
   * pair and feature on the vector ALUs, as the paper prescribes for these
   * blocks (Sec. 4.3).  Results are bit-identical with and without it. */
  GLA_FLAG_FP32_DIAGONAL = 1u << 2,
  /* Bits 8..11 select a single stage of an entry point's launch sequence (0 =
   * the whole sequence), so that a profiler or benchmark can time each kernel
   * on its own stream with events.  Running the stages 1, 2, ... in order with
   * the same arguments and workspace gives exactly the result of stage 0.
   *   gla_chunk_fwd: 1 = gate factors, gated operands and intra-chunk P
   *                  2 = state pass and chunk outputs
   *   gla_chunk_bwd: 1 = as forward stage 1 (skipped with REUSE_FWD_WORKSPACE)
   *                  2 = forward sweep over key-feature tiles: dq_inter
   *                      (and dP = (dO V^T) (.) M)
   *                  3 = intra-chunk terms, chunk-parallel: dq, and dk_intra
   *                      and its share of the gate gradient for stage 4
   *                  4 = reverse sweep over key-feature tiles: dk, dlog_alpha
   *                  5 = reverse sweep over value-column tiles: dv, dS0
   * Out-of-range stage numbers return GLA_ERR_SHAPE. */
  GLA_STAGE_SHIFT = 8,
  GLA_STAGE_MASK = 0xFu << 8,
  /* Bits 16..30 fix the number of sequence segments per head of the chunkwise
   * calls (the split described under "Few heads, long sequences" above)
   * instead of letting the shape decide; 0 = decided from the shape.  This is
   * the choice of Sec. 3.3 between keeping the chunk-level states on chip and
   * materializing them in HBM: 1 keeps each head's state in the workgroups
   * for the whole sequence (the non-materialization version: no state is
   * written), T/C (one chunk per segment) writes every chunk's initial state
   * S_[n] to the workspace and computes all chunks in parallel (the
   * materialization version), and a value in between materializes the state
   * at the start of every (T/C)/n-th chunk.  The value must divide T/C, T
   * must be a multiple of C (when T > 0), and B*H times the value must not
   * exceed 65535; else GLA_ERR_UNSUPPORTED (and gla_workspace_bytes gives
   * 0).  gla_workspace_bytes honours it (the states take
   * 2 B H n d_k d_v fp32 in the forward's workspace, one more such array in
   * the backward's); a forward and the backward that reuses its workspace
   * must be given the same value.  The general form accepts only 0 and 1;
   * the recurrent calls ignore it.  GLA_SEGMENTS(n) builds the field. */
  GLA_SEGMENTS_SHIFT = 16,
  GLA_SEGMENTS_MASK = 0x7FFF << 16
};
#define GLA_SEGMENTS(n) ((uint32_t)(n) << GLA_SEGMENTS_SHIFT)

typedef struct {
  int32_t B, H;      /* batch rows and heads; heads are independent            */
  int32_t T;         /* sequence length L                                      */
  int32_t dk, dv;    /* per-head key/value widths d'_k, d'_v (Sec. 4.4)        */
  int32_t chunk;     /* chunk length C (Sec. 2.2)                              */
  int32_t subchunk;  /* sub-chunk length c of the secondary tiling (Sec. 4.3)  */
  int32_t io;        /* gla_dtype of every non-state tensor                    */
  uint32_t flags;    /* GLA_FLAG_* bits                                        */
  float gate_tau;    /* 0: the log_alpha argument holds log alpha.  tau > 0:
                      * it holds the gate pre-activation z of the GLA gate
                      * alpha = sigmoid(z)^(1/tau) (Sec. 4.4; the paper uses
                      * tau = 16), applied on the fly wherever log alpha is
                      * read, and the backward's dlog_alpha output receives
                      * dL/dz = dL/dlog_alpha * sigmoid(-z) / tau.  Negative,
                      * infinite or NaN values return GLA_ERR_SHAPE.         */
} gla_problem;

/* Bytes of device workspace gla_chunk_fwd (op = 0), gla_chunk_bwd (op = 1)
 * or gla_chunk_bwd_general (op = 2) needs for this problem; 0 if the problem
 * is invalid.  Each layout begins with the previous one, so a buffer sized
 * for a larger op can be passed to the smaller ones (required for
 * GLA_FLAG_REUSE_FWD_WORKSPACE; gla_chunk_fwd_general uses op 0's). */
size_t gla_workspace_bytes(const gla_problem *prob, int op);

/* Forward, chunkwise form (Sec. 4.2 / 4.3; the non-materialized state pass of
 * Sec. 3.3 and App. B, Alg. 5, with the intra-chunk part of Alg. 3).
 *   in : q, k, v, log_alpha (nullable); S0 (nullable, fp32)
 *   out: o; S_T (nullable, fp32, the state after the last step)
 *   workspace: device buffer of at least gla_workspace_bytes(prob, 0) bytes;
 *   on return its contents are what GLA_FLAG_REUSE_FWD_WORKSPACE expects. */
gla_status gla_chunk_fwd(const gla_problem *prob, const void *q, const void *k, const void *v,
                         const void *log_alpha, const float *S0, void *o, float *S_T,
                         void *workspace, size_t workspace_bytes, void *stream);

/* gla_chunk_fwd without any allocation, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, results (bit for bit) and kernels
 * as gla_chunk_fwd, minus the workspace: the library uses a fixed device
 * array of GLA_NOALLOC_SCRATCH_BYTES bytes in its code object instead, which
 * every GPU the library runs on holds from the library's load until the
 * process ends.  The caller still provides every input and output buffer.
 * Problems whose forward workspace (gla_workspace_bytes(prob, 0)) exceeds
 * that size return GLA_ERR_SCRATCH before anything is enqueued.  The call
 * allocates, frees and clears nothing; its first call on a device looks up
 * that device's address of the array (hipGetSymbolAddress).  Every call on
 * one GPU uses that GPU's one array, so calls whose work overlaps on a GPU
 * (other streams, other host threads) race and give undefined results;
 * calls ordered on one stream are safe.  The array keeps the last call's
 * contents, which no call reads before writing. */
#define GLA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)
gla_status gla_chunk_fwd_noalloc(const gla_problem *prob, const void *q, const void *k, const void *v,
                                 const void *log_alpha, const float *S0, void *o, float *S_T, void *stream);

/* Backward of gla_chunk_fwd for the loss L = sum(o * dO) + sum(S_T * dS_T)
 * (App. B, Alg. 4/6 with the closed-form gate gradient of Sec. 4.3):
 *   dq, dk, dv: gradients of q, k, v;
 *   dlog_alpha: gradient w.r.t. log_alpha, = revcumsum(q*dq - k*dk)
 *               + rowsum(S_T * dS_T) (the last term vanishes when dS_T = 0);
 *   dS0 (nullable): gradient w.r.t. S0.
 *   in : q, k, v, log_alpha (nullable), S0 (nullable), dO, dS_T (nullable)
 *   workspace: at least gla_workspace_bytes(prob, 1) bytes. */
gla_status gla_chunk_bwd(const gla_problem *prob, const void *q, const void *k, const void *v,
                         const void *log_alpha, const float *S0, const void *dO,
                         const float *dS_T, void *dq, void *dk, void *dv, void *dlog_alpha,
                         float *dS0, void *workspace, size_t workspace_bytes, void *stream);

/* Forward in the recurrent form (Sec. 4.1, Eq. 3), one step at a time with the
 * state in fp32; no workspace.  prob->chunk and prob->subchunk are ignored.
 *   in : q, k, v, log_alpha (nullable); S0 (nullable)   out: o; S_T (nullable) */
gla_status gla_recurrent_fwd(const gla_problem *prob, const void *q, const void *k,
                             const void *v, const void *log_alpha, const float *S0, void *o,
                             float *S_T, void *stream);

/* General gated form (App. C): G_t = alpha_t^T beta_t with a value-side gate
 * beta_t in (0, 1]^{d_v} besides the key-side alpha_t,
 *     S_t = (alpha_t^T beta_t) (.) S_{t-1} + k_t^T v_t,   o_t = q_t S_t.
 * log_beta: [B, H, T, d_v] (io dtype), finite and <= 0; NULL means beta = 1,
 * which is exactly gla_chunk_fwd / gla_recurrent_fwd.  Every other argument,
 * flag (scalar key gate, gate_tau on the key gate) and the workspace are as
 * for those calls.  The chunkwise form normalises the value side per chunk:
 * the decay of beta accumulated over one chunk of one value column,
 * -sum log beta, must stay below ~80, else outputs overflow (a shorter chunk
 * widens the range; the recurrent form has no such limit). */
gla_status gla_chunk_fwd_general(const gla_problem *prob, const void *q, const void *k, const void *v,
                                 const void *log_alpha, const void *log_beta, const float *S0, void *o,
                                 float *S_T, void *workspace, size_t workspace_bytes, void *stream);
gla_status gla_recurrent_fwd_general(const gla_problem *prob, const void *q, const void *k,
                                     const void *v, const void *log_alpha, const void *log_beta,
                                     const float *S0, void *o, float *S_T, void *stream);

/* Backward of gla_chunk_fwd_general for L = sum(o * dO) + sum(S_T * dS_T):
 * the outputs of gla_chunk_bwd plus dlog_beta ([B, H, T, d_v], nullable) =
 * revcumsum(o * dO - v * dv) + colsum(S_T * dS_T) (App. C), which needs the
 * forward's output o (required when dlog_beta is wanted).  log_beta is
 * required here.  The key gate may be scalar (GLA_FLAG_SCALAR_GATE) but not
 * the gate epilogue (gate_tau > 0: GLA_ERR_UNSUPPORTED).  Workspace: at least
 * gla_workspace_bytes(prob, 2) bytes; GLA_FLAG_REUSE_FWD_WORKSPACE as for
 * gla_chunk_bwd.  Stage selector: 1 = key-gate factors (as gla_chunk_bwd),
 * 2 = value-gate operands, 3 = dq sweep, 4 = intra-chunk terms, 5 = dk sweep,
 * 6 = dv sweep, 7 = the value-gate gradient. */
gla_status gla_chunk_bwd_general(const gla_problem *prob, const void *q, const void *k, const void *v,
                                 const void *log_alpha, const void *log_beta, const float *S0, const void *o,
                                 const void *dO, const float *dS_T, void *dq, void *dk, void *dv,
                                 void *dlog_alpha, void *dlog_beta, float *dS0, void *workspace,
                                 size_t workspace_bytes, void *stream);

/* Output side of the layer (Sec. 4.4): per head and row, y_t = Swish(g_t) (.)
 * LN(o_t) with LN(x) = w (.) (x - mean(x)) / sqrt(var(x) + eps) + b over the
 * d_v features of one head (biased variance), g the output-gate
 * pre-activation (its projection is the caller's GEMM).
 * prob: only B, H, T, dv and io are used (dv a multiple of 16, <= 1024).
 *   o, g, y, dy, d_o, dg : [B, H, T, d_v] (io dtype)
 *   ln_w, ln_b, dln_w, dln_b : [H, d_v] fp32, nullable (absent w = 1, b = 0;
 *                              an absent gradient is not computed)
 *   stats (nullable, fp32 [B, H, T, 2]): mean and 1/sqrt(var + eps) per row
 *   eps: finite and > 0, else GLA_ERR_SHAPE.
 * The backward (loss L = sum(y * dy)) recomputes the row statistics; its
 * workspace holds per-(batch row, head, 64-step block) partial sums of the
 * affine gradients (gla_output_gate_workspace_bytes; may be 0 bytes / NULL
 * when dln_w and dln_b are both NULL or there are no rows; smaller than
 * needed: GLA_ERR_WORKSPACE).  With no rows the affine gradients are written
 * as zeros.  The affine gradients are summed in a fixed order, so repeated
 * calls give the same bits.  d_o is the dO of gla_chunk_bwd. */
size_t gla_output_gate_workspace_bytes(const gla_problem *prob);
gla_status gla_output_gate_fwd(const gla_problem *prob, const void *o, const void *g,
                               const float *ln_w, const float *ln_b, float eps, void *y,
                               float *stats, void *stream);
gla_status gla_output_gate_bwd(const gla_problem *prob, const void *o, const void *g,
                               const float *ln_w, const float *ln_b, float eps, const void *dy,
                               void *d_o, void *dg, float *dln_w, float *dln_b, void *workspace,
                               size_t workspace_bytes, void *stream);

/* Static, human-readable name of a status code (never NULL). */
const char *gla_status_string(gla_status status);

#ifdef __cplusplus
}
#endif

#endif /* GLA_H_ */
