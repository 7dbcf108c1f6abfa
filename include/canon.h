/*
 * canon.h - C ABI of libcanon: one replayed training step in canonical order, on MI355X (gfx950).
 *
 * The method is the paper's auditable replay:
 *   - every floating-point reduction follows one fixed order on all hardware (section "Reproducible
 *     Operations": fixed reduction order, one fused-multiply-add convention, subnormals flushed);
 *   - the gradients of the data-parallel ranks are combined by Algorithm 1 (audit replay of one step),
 *     with Algorithm 2 (binary-carry tree fold) across replicas, the ascending-shard reduce-scatter order
 *     and averages taken as reciprocal multiplies (appendix "Deterministic Gradient Reduction");
 *   - AdamW is widened to fp32 and rounded to bf16 once (training recipe, optimizer-state precision).
 * The order itself (rules R0-R12, "CANON-v1") is stated with each entry point below.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE memory owned by the caller.  bf16 tensors are uint16_t bit patterns.
 *     Arrays of tensor pointers (e.g. the parameter list) are HOST arrays of device pointers, read during
 *     the call.  Structs are passed by host pointer and read during the call.
 *   - The library allocates no device memory.  Scratch space comes from a caller-owned workspace whose
 *     size is given by the matching *_workspace_bytes function.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).  Work is enqueued on it and
 *     the call returns after validation and launch; device faults surface at the caller's next
 *     synchronisation.
 *   - Invalid arguments return CANON_EINVAL and enqueue nothing.  Valid requests outside what this
 *     version implements return CANON_EUNSUPPORTED.  A failed launch returns CANON_EDEVICE.
 *   - Calls on different streams may run concurrently; calls that share output buffers must be ordered
 *     by the caller.
 */
#ifndef CANON_H
#define CANON_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  CANON_OK = 0,
  CANON_EINVAL = -1,
  CANON_EUNSUPPORTED = -2,
  CANON_EDEVICE = -3,
  CANON_EWORKSPACE = -4
} canon_status;

/* The declared order.  Version 1 requires: version = 1, chunk = 32, tree = CANON_TREE_BINARY_CARRY,
   ftz = 1.  Anything else returns CANON_EUNSUPPORTED. */
enum { CANON_TREE_BINARY_CARRY = 0 };
typedef struct {
  int32_t version; /* 1 */
  int32_t chunk;   /* chain length: 32 */
  int32_t tree;    /* CANON_TREE_BINARY_CARRY (Algorithm 2 over chunk partials) */
  int32_t ftz;     /* 1: subnormal inputs read as signed zero; tiny results (after rounding) flushed */
} canon_order;

/* Algorithm 1's mesh: N = dp_shard * dp_replicate virtual ranks, rank r = rep * dp_shard + shard,
   each accumulating `accum` microbatches. */
typedef struct {
  int32_t accum, dp_shard, dp_replicate;
} canon_dp_plan;

/* Llama-style decoder: pre-norm RMSNorm blocks, causal attention with half-split RoPE, SwiGLU MLP (gate
   and up as one fused weight), untied embedding and head, no biases (the paper's architecture section).
   The paper's further variants (R16, same section) are switched on by the fields after rms_eps; all zero
   gives the plain block:
     n_kv_heads:     0 (= n_heads) or a divisor of n_heads; query head h reads key/value head
                     h / (n_heads / n_kv_heads).  w_qkv is [(n_heads + 2 n_kv_heads) head_dim, d_model]:
                     query heads, then key heads, then value heads.  The gradient of a shared key (value)
                     head is one contraction over its group's query heads (ascending) and their queries.
     qk_norm:        1: gain-free RMSNorm (eps = rms_eps) of every q and k head row before the rotation,
                     its output kept fp32 into the rotation.
     embed_norm:     1: an RMSNorm with its own gain (tensor "embed_norm", after embed in the declared
                     order) on the gathered embedding rows, fp32 output into the first block.
     swa_window:     0: every layer full causal; W > 0: query i sees keys i - W < j <= i in every layer
                     except every swa_full_every-th (l + 1 a multiple of it, 0 = none) and the last.
     z_loss:         weight of the z-loss (0: none): row loss RN(CE + RN(z * RN(lse^2))), probabilities
                     scaled by RN(1 + RN(RN(2 z) * lse)) in the logit gradient.
   The attention kernels of the paper's int8 path (training-details paragraph on int8 computation):
     pv_int8:        1: the forward P.V in int8 per block (R17, canon_attn_pv_i8 below); head_dim a multiple of
                     32 up to 256 and seq <= 8192, else CANON_EUNSUPPORTED.  The backward stays the bf16 one
                     (straight-through).
     dq_fixed_bits:  0: dQ by the canonical GEMM; F in [1, 62]: dQ accumulated in 64-bit fixed point with F
                     fractional bits (R18, canon_attn_dq_fixed below); head_dim in {16, 32, 64, 128}.
     int8_linear:    1: the four projections of every block (q/k/v, output, gate/up, down) in int8 (R19, the
                     paper's W8A8 quantisation-aware training): weights quantised with their per-row steps
                     re-pinned from the weights (canon_quant_scales), the bf16 input with a learned
                     per-tensor activation step, the exact int8 product dequantised (canon_gemm_i8); the
                     backward is canon_qlinear_bwd on the widened bf16 upstream gradient, and each activation
                     step s gets LSQ's gradient RN(R1_{t,k} RN(dx * delta) * RN32(1/sqrt(127 K))) with
                     delta = -128 / 127 outside the integer range and RN(rne(v) - v) inside (v = RN(x / s);
                     0 for a step that is not > 0).  Each layer then has four more tensors after w_down, the
                     bf16 activation steps sx_qkv, sx_o, sx_gate_up, sx_down (one element each, no weight
                     decay).  Needs the tokens per call, d_model, 2 d_ffn and the q/k/v width to be multiples
                     of 256 (whole rotation blocks), else CANON_EUNSUPPORTED. */
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab, seq, micro_seqs;
  float rms_eps; /* fp32 value, e.g. RN32(1e-5) */
  int32_t n_kv_heads, qk_norm, embed_norm, swa_window, swa_full_every;
  float z_loss;
  int32_t pv_int8, dq_fixed_bits;
  int32_t int8_linear;
} canon_model_cfg;

/* AdamW constants, each evaluated in double and rounded once to fp32 by the caller (R9). */
typedef struct {
  float lr, beta1, one_minus_beta1, beta2, one_minus_beta2, inv_bc1, inv_bc2, eps, decay_factor;
} canon_adamw_consts;

/* ------------------------------------------------------------------------------------------------ */
/* GEMM (R1, R2).  C[i,j] = sum over k of A(i,k) B(k,j), bf16 operands, fp32 result.  The k terms are
   cut into chunks of 32, each a left-to-right fma chain from +0 in ascending k, and the chunk partials
   are combined by Algorithm 2 (binary carry, leftover blocks smallest first).  A(i,k) = a[i*lda + k]
   (trans_a = 0) or a[k*lda + i] (trans_a = 1); B(k,j) = b[k*ldb + j] (trans_b = 0) or b[j*ldb + k]
   (trans_b = 1); C row-major with leading dimension ldc >= n.  k = 0 writes +0; m = 0 or n = 0 is a
   no-op.  Operands must not alias C.
   epilogue: NULL or kind CANON_EPI_NONE writes C = d (the canonical sum d above).  kind CANON_EPI_ACCUM_PLAN
   (Algorithm 1's microbatch accumulation, with every average a multiply by a reciprocal as the appendix on
   deterministic gradient reduction states it): C = RN(C + RN(d * scale)), C read and written in place; with
   C cleared to +0 before the first microbatch and scale = RN32(1/accum), accum calls leave C = g_r of the
   plan (R7).  Another kind returns CANON_EINVAL. */
enum { CANON_EPI_NONE = 0, CANON_EPI_ACCUM_PLAN = 1 };
typedef struct {
  int32_t kind;
  float scale;
} canon_gemm_epilogue;
canon_status canon_gemm(const canon_order* order, int32_t trans_a, int32_t trans_b, int64_t m, int64_t n,
                        int64_t k, const uint16_t* a, int64_t lda, const uint16_t* b, int64_t ldb, float* c,
                        int64_t ldc, const canon_gemm_epilogue* epilogue, void* stream);

/* Strided batched form: matrix z of the batch uses a + z*stride_a, b + z*stride_b, c + z*stride_c
   (strides in elements). */
canon_status canon_gemm_strided_batched(const canon_order* order, int32_t trans_a, int32_t trans_b, int64_t m,
                                        int64_t n, int64_t k, const uint16_t* a, int64_t lda, int64_t stride_a,
                                        const uint16_t* b, int64_t ldb, int64_t stride_b, float* c, int64_t ldc,
                                        int64_t stride_c, int64_t batch, void* stream);

/* ------------------------------------------------------------------------------------------------ */
/* RMSNorm rows (R3; the architecture section's pre-norm RMSNorm without bias), x fp32 [rows, cols].
   dir = CANON_FWD: y (bf16 [rows, cols]) = bf16(RN(RN(x*r)*g)) with r = CRdiv(1, CRsqrt(RN(ms + eps))),
       ms = RN(R1(x*x) * RN(1/cols)); rstd (fp32 [rows]) = r.  dy, dx, dgain unused (may be NULL).
   dir = CANON_BWD: inputs x, gain, rstd (from the forward), dy (fp32 [rows, cols]); outputs dx (fp32
       [rows, cols]) and, if dgain != NULL, dgain (fp32 [cols]) = R1 over rows of RN(dy*RN(x*r)).
       dx also serves as scratch for the dgain chunk partials before it receives its values, so dx must not
       overlap x, dy, rstd, gain or dgain (CANON_EINVAL otherwise).
   dir = CANON_FWD_F32: as CANON_FWD with y fp32 [rows, cols] = RN(RN(x*r)*g) (no bf16 rounding; the
       embedding norm of R16). */
enum { CANON_FWD = 0, CANON_BWD = 1, CANON_FWD_F32 = 2 };
canon_status canon_rownorm(const canon_order* order, int32_t dir, int64_t rows, int64_t cols, const float* x,
                           const uint16_t* gain, float eps, void* y, float* rstd, const float* dy, float* dx,
                           float* dgain, void* stream);

/* ------------------------------------------------------------------------------------------------ */
/* Row softmax / cross-entropy (R5, R6; the audit section names the sums inside softmax among the
   reductions that need a definite order).
   mode = CANON_SOFTMAX_CAUSAL: x = fp32 raw scores [rows, cols] forming rows/cols stacked square
       matrices; row r is query i = r mod cols.  score = RN(x*scale); keys j <= i only, and with
       window > 0 only keys j > i - window (R16's sliding window); the row sum still runs over every key
       position, masked ones as +0 terms.  out = probabilities bf16 [rows, cols], +0 for masked keys.
       targets, inv_tokens, z_loss, row_loss, mean_loss unused.
   mode = CANON_XENT: x = bf16 logits [rows, cols = vocab]; targets int32 [rows] in [0, cols);
       out = dlogits bf16 [rows, cols] = bf16(RN(RN(p' - onehot) * inv_tokens)) with p' = p, or with
       z_loss > 0 p' = RN(p * RN(1 + RN(RN(2 z_loss) * lse))); row_loss fp32 [rows] = RN(lse - x[target]),
       plus RN(z_loss * RN(lse * lse)) with the z-loss; mean_loss (fp32 scalar, device) =
       RN(R1(row_loss) * inv_tokens).  Targets are checked on the device; an out-of-range target makes
       its row loss, and so mean_loss, NaN.  window unused.
   window >= 0, z_loss >= 0 and finite (CANON_EINVAL otherwise). */
enum { CANON_SOFTMAX_CAUSAL = 0, CANON_XENT = 1 };
canon_status canon_softmax_xent(const canon_order* order, int32_t mode, int64_t rows, int64_t cols, const void* x,
                                float scale, int64_t window, const int32_t* targets, float inv_tokens, float z_loss,
                                uint16_t* out, float* row_loss, float* mean_loss, void* stream);

/* ------------------------------------------------------------------------------------------------ */
/* Gradient plan (R7 = Algorithm 1 with Algorithm 2 over replicas, averages by reciprocal multiply).
   grads: HOST array of N*accum device pointers (N = dp_shard*dp_replicate), rank-major, microbatch-
   minor (grads[r*accum + k]); each points to n fp32 values.  out: n fp32 values.  This version fuses
   up to 64 buffers in one pass (CANON_EUNSUPPORTED beyond). */
canon_status canon_grad_accum(const canon_order* order, const canon_dp_plan* plan, int64_t n,
                              const float* const* grads, float* out, void* stream);

/* The same plan fed one microbatch gradient at a time (Algorithm 1's loop, with Algorithm 2's stack over the
   replicas), so that it can stop after any microbatch and resume later, in another process or in other
   memory: the analogue of restarting a run from its last checkpoint and comparing the repeated steps'
   hashes (the paper's training-run account).  canon_step runs its plan through this same code.
   The whole state is a plain host record (canon_plan_cursor: the plan, n, the count of microbatches in,
   the stack's levels and slot numbers; no pointers) plus a caller-owned device buffer of
   canon_plan_state_bytes(plan, n) bytes (256-byte aligned) holding the partial sums in slots of n floats.
   To persist: copy the record and the buffer's bytes; to resume: copy both back, into any buffer of that
   size.  canon_plan_begin initialises the record (host only).  canon_plan_push takes the gradient of the
   next microbatch in Algorithm 1's order, rank-major and microbatch-minor (rank r = next / accum,
   microbatch k = next % accum): grad, n fp32 device values, read only.  canon_plan_finish, after all
   N*accum pushes, writes the reduced gradient to out (n fp32, device); it leaves the buffer's contents
   unspecified.  Both return CANON_EINVAL for a record that the calls above cannot produce (position out
   of range, a stack shape or a shard sum that does not match the position, slots repeated or out of
   range), a push after the last microbatch or a finish before it, and leave the record unchanged on any
   error.  The result is bit-identical to canon_grad_accum over the same buffers, wherever the plan was
   stopped and resumed.  dp_replicate below 2^31. */
#define CANON_PLAN_MAX_DEPTH 31
typedef struct {
  canon_dp_plan plan;
  int32_t next;                          /* microbatches pushed */
  int64_t n;                             /* floats per gradient */
  int32_t inner;                         /* slot of the current replica's shard sum, -1 when none */
  int32_t depth;                         /* entries on Algorithm 2's stack */
  int32_t level[CANON_PLAN_MAX_DEPTH];   /* level of entry i, bottom first (strictly decreasing) */
  int32_t slot[CANON_PLAN_MAX_DEPTH];    /* slot holding entry i */
} canon_plan_cursor;
size_t canon_plan_state_bytes(const canon_dp_plan* plan, int64_t n);
canon_status canon_plan_begin(const canon_dp_plan* plan, int64_t n, canon_plan_cursor* cursor);
canon_status canon_plan_push(const canon_order* order, canon_plan_cursor* cursor, const float* grad, void* state,
                             size_t state_bytes, void* stream);
canon_status canon_plan_finish(const canon_order* order, canon_plan_cursor* cursor, void* state, size_t state_bytes,
                               float* out, void* stream);

/* ------------------------------------------------------------------------------------------------ */
/* AdamW (R9): per tensor t of n_tensors (HOST arrays of device pointers and host sizes), widen the bf16
   parameter, apply decoupled decay if decay_mask[t] (host) != 0, update fp32 m and v, bias-correct by
   reciprocal multiply, divide by RN(CRsqrt(vh) + eps), round the parameter to bf16 once.  In place. */
canon_status canon_adamw(int64_t n_tensors, const int64_t* sizes, uint16_t* const* params, float* const* m,
                         float* const* v, const float* const* grads, const uint8_t* decay_mask,
                         const canon_adamw_consts* consts, void* stream);

/* ------------------------------------------------------------------------------------------------ */
/* Global-norm clip and spike skip (R15; the optimizer paragraph of the training setup clips gradients to a
   global l2 norm of 1.0, and the section on gradient behaviour skips five optimizer steps when the
   pre-clip norm exceeds 5).
   The gradient tensors laid end to end in the given order form one vector g; its pre-clip norm is
   CRsqrt(Q), Q the R1 sum over g's flat index of RN(g_i * g_i) (chunks of 32 run across tensor
   boundaries).  coef = CRdiv(max_norm, RN(norm + RN32(1e-6))); when coef < 1 every element becomes
   RN(g_i * coef), otherwise g is left untouched.  A norm that is not <= spike_norm (NaN included) is a
   spike: it sets *skip_state to skip_steps.  The step applies no update when *skip_state > 0 after that,
   and such a step takes one off *skip_state; so one spike skips the spiking step and the skip_steps - 1
   after it, and a spike inside that window starts it again.
   Settings and outputs (all pointers device memory, written in stream order):
     max_norm > 0 (+inf: no clip); spike_norm; skip_steps >= 0 (0: no spike rule, skip_state unused);
     norm_out: fp32 scalar, the pre-clip norm, or NULL; skip_state: int32 counter, read and written,
     required when skip_steps > 0 (start it at 0); skipped_out: int32, 1 when this step applies no update,
     or NULL.  Invalid settings: CANON_EINVAL. */
typedef struct {
  float max_norm;
  float spike_norm;
  int32_t skip_steps;
  float* norm_out;
  int32_t* skip_state;
  int32_t* skipped_out;
} canon_clip;

/* Norm, spike decision and clip of n_tensors fp32 device buffers (grads[t] of sizes[t] elements, sizes[t]
   >= 0; the clip writes them in place).  The caller skips its optimizer update when *skipped_out is 1.
   workspace: device memory of canon_clip_grad_norm_workspace_bytes(n_tensors, sizes) bytes, 256-byte
   aligned; it holds the tensor table and the block sums.  Up to 2^40 elements in total. */
canon_status canon_clip_grad_norm(const canon_order* order, int64_t n_tensors, const int64_t* sizes,
                                  float* const* grads, const canon_clip* clip, void* workspace,
                                  size_t workspace_bytes, void* stream);
size_t canon_clip_grad_norm_workspace_bytes(int64_t n_tensors, const int64_t* sizes);

/* ------------------------------------------------------------------------------------------------ */
/* One decoder block, forward then backward, for `batch` sequences of cfg->seq tokens (T = batch*seq).
   x, dy: fp32 [T, d_model] (block input, gradient of the block output).  w: HOST array of the six bf16
   block tensors in the order attn_norm [d], w_qkv [(n_heads + 2 n_kv_heads) head_dim, d], w_o [d, d],
   ffn_norm [d], w_gate_up [2F, d] (gate rows first), w_down [d, F], then with int8_linear the four bf16
   activation steps [1] (ten tensors; dw likewise).  The block's attention window is
   cfg->swa_window (the step applies the per-layer rule); embed_norm and z_loss do not apply to a block.  rope_cos/rope_sin: fp32 [seq, head_dim/2].  Outputs: y (block
   output), dx (input gradient), dw: HOST array of six fp32 gradient buffers shaped like w. */
canon_status canon_block_fwd_bwd(const canon_order* order, const canon_model_cfg* cfg, int32_t batch,
                                 const float* x, const float* dy, const uint16_t* const* w, const float* rope_cos,
                                 const float* rope_sin, float* y, float* dx, float* const* dw, void* workspace,
                                 size_t workspace_bytes, void* stream);
size_t canon_block_workspace_bytes(const canon_model_cfg* cfg, int32_t batch);

/* ------------------------------------------------------------------------------------------------ */
/* One training step (Algorithm 1 on one device).  For each virtual rank r in mesh order and each of its
   `accum` microbatches (R12: rank r owns windows m with m mod N == r, micro_seqs consecutive ones per
   microbatch), run forward and backward of the whole model, then reduce the gradients and the
   microbatch losses through the plan and apply AdamW (R9).
   params, m, v: HOST arrays of n = 3 + 6*n_layers (10*n_layers with int8_linear; +1 with embed_norm) device
   pointers in the declared order: embed [V, d]; [embed_norm [d]]; per layer attn_norm, w_qkv, w_o,
   ffn_norm, w_gate_up, w_down [, sx_qkv, sx_o, sx_gate_up, sx_down]; final_norm [d]; head [V, d].  params
   (bf16), m and v (fp32) are updated in place.  windows: device int32 [M, seq+1], M = N*accum*
   micro_seqs, each token in [0, vocab) (checked on the device: an out-of-range token makes the loss
   NaN and leaves the parameters unchanged).  loss_out: device fp32 scalar.  grads_out: NULL, or a HOST
   array of n device fp32 buffers that receive the reduced gradient (before any clip).  clip: NULL, or the
   R15 settings (canon_clip above) applied to the reduced gradient of all n tensors in the declared order
   between the plan and AdamW; a skipped step leaves params, m and v unchanged.  An out-of-range token
   also makes *norm_out NaN and sets *skipped_out, and leaves *skip_state unchanged.  step_t: AdamW's step
   index t >= 1 (else CANON_EINVAL) that consts was computed for; the bias corrections RN32(1/(1 - beta^t))
   come in consts (evaluated by the caller in binary64 and rounded once), so the library uses t only for this
   check; a caller that skips an update does not advance t.
   state_digest: NULL, or device memory of 32 bytes that receives the per-step audit hash (the paper's
   state-hash appendix: every step digests its data batch, parameters, optimizer state and gradients):
   H1 (canon_state_hash below) over, in this order, windows (M*(seq+1) int32), the n parameters (bf16) and
   the n tensors of m and of v (fp32) as this step leaves them, and the n tensors of the reduced gradient
   (fp32, before any clip), each in the declared order.  The digest names the tensors, not the plan's
   shards, so it is the same for every plan that gives the same bits.  The workspace must then be 256-byte
   aligned (CANON_EINVAL otherwise); canon_step_workspace_bytes includes the hash's tables. */
canon_status canon_step(const canon_order* order, const canon_model_cfg* cfg, const canon_dp_plan* plan,
                        uint16_t* const* params, float* const* m, float* const* v, int32_t step_t,
                        const int32_t* windows, const float* rope_cos, const float* rope_sin,
                        const canon_adamw_consts* consts, const canon_clip* clip, void* workspace,
                        size_t workspace_bytes, float* loss_out, float* const* grads_out, uint8_t* state_digest,
                        void* stream);
size_t canon_step_workspace_bytes(const canon_model_cfg* cfg, const canon_dp_plan* plan);

/* ------------------------------------------------------------------------------------------------ */
/* ------------------------------------------------------------------------------------------------ */
/* int8 quantised linear, forward (the paper's W8A8 training path: the architecture section's int8
   quantisation-aware training bullet, the training-details paragraph on int8 computation, and the
   appendix that replaces the learned weight step by its re-pinned LSQ initialisation value).

   canon_quant_scales: per-row step of a bf16 weight matrix w [rows, cols] (one row per output channel):
     scale[r] = RN(RN(2 * RN(R1(|w[r,:]|) * RN(1/cols))) * RN(1/sqrt(127))), R1 over the row in column
     order.  scale: device fp32 [rows].  cols in [1, 32768].
   canon_quantize: q = clamp(rne(RN(x / s)), -128, 127) element by element for x [rows, cols] fp32
     (in_dtype CANON_F32) or bf16 (CANON_BF16); s = scale[r] for row r when per_row, else scale[0]
     (e.g. a per-tensor activation step).  A step that is not > 0 once flushed, or a NaN quotient, gives
     0.  scale, x, q: device memory; q int8 [rows, cols].
   canon_gemm_i8: acc[i][j] = sum_k a[i][k] * b[j][k] exactly, a int8 [m, k] (leading dim lda), b int8
     [n, k] (ldb; one output column per row, as weights [out][in]); writes acc (int32, may be NULL) and
     y[i][j] = RN(RN(RN32(acc) * sa[0]) * sb[j]) (fp32, may be NULL; sa device scalar, sb device [n]),
     both with leading dim ldc.  k in [0, 65536] keeps |acc| < 2^31.  The integer sum is exact in any
     order, so this kernel runs on the int8 matrix instructions without an order constraint. */
enum { CANON_F32 = 0, CANON_BF16 = 1 };
canon_status canon_quant_scales(const canon_order* order, int64_t rows, int64_t cols, const uint16_t* w,
                                float* scale, void* stream);
canon_status canon_quantize(int64_t rows, int64_t cols, int32_t in_dtype, const void* x, const float* scale,
                            int32_t per_row, int8_t* q, void* stream);
canon_status canon_gemm_i8(int64_t m, int64_t n, int64_t k, const int8_t* a, int64_t lda, const int8_t* b,
                           int64_t ldb, int32_t* acc, float* y, int64_t ldc, const float* sa, const float* sb,
                           void* stream);

/* Backward of the int8 quantised linear (the same training-details paragraph: straight-through
   estimator, both gradient GEMMs in int8 after a Walsh-Hadamard rotation along the contraction
   dimension).  Inputs: dy fp32 [T, N]; the forward's codes qx int8 [T, K] with the device scalar step sx
   and qw int8 [N, K] with the device steps sw [N].  Outputs (either may be NULL): dx fp32 [T, K] =
   dy . W^ and dw fp32 [N, K] = dy^T . X^, where W^ = RN(sw[n] * qw), X^ = RN(sx * qx).  Each operand is
   rotated along the contraction dimension (N for dx, T for dw; a multiple of 256 when that output is
   asked for) in blocks of 256 by the Sylvester matrix scaled by 1/16 (fast transform, strides 1..128),
   quantised with the per-tensor step RN(amax * RN(1/127)) (amax: the largest |value| by bit pattern),
   multiplied exactly on the int8 matrix cores and dequantised as RN(RN(RN32(acc) * s_left) * s_right).
   workspace: device memory of canon_qlinear_bwd_workspace_bytes(T, N, K) bytes (the rotated operands'
   codes; the rotated values themselves are recomputed, never stored); T*N and K*max(N, T) at most 2^34. */
canon_status canon_qlinear_bwd(const canon_order* order, int64_t T, int64_t N, int64_t K, const float* dy,
                               const int8_t* qx, const float* sx, const int8_t* qw, const float* sw, float* dx,
                               float* dw, void* workspace, size_t workspace_bytes, void* stream);
size_t canon_qlinear_bwd_workspace_bytes(int64_t T, int64_t N, int64_t K);

/* ------------------------------------------------------------------------------------------------ */
/* Canonical state hash H1 (the paper's per-step state hash, moved onto the device as the paper proposes;
   the paper leaves the function open, so H1 is this library's definition): SHA-256 (FIPS 180-4) over a
   fixed tree.  A tensor of n bytes is cut into nb = ceil(n/64) blocks of 64 bytes and W = max(1,
   ceil(nb/1024)) leaves, leaf l holding blocks l, l+W, l+2W, ... in order; leaf digest = SHA-256 of its
   bytes; leaf digests fold pairwise level by level as SHA-256(left || right), an odd last node passing up
   unchanged; tensor digest = SHA-256(0x02 || index (8 bytes LE) || n (8 bytes LE) || root); state digest =
   SHA-256(0x03 || tensor digests in order).
   ptrs, nbytes: HOST arrays of n_tensors device pointers and byte counts (any tensors: parameters, moments,
   gradients, batches).  digest: device, 32 bytes.  workspace: device memory of
   canon_state_hash_workspace_bytes(n_tensors, nbytes) bytes, 256-byte aligned.  The call stages a small
   table from host memory into the workspace (copied before it returns) and enqueues three kernels. */
canon_status canon_state_hash(int64_t n_tensors, const void* const* ptrs, const int64_t* nbytes, uint8_t* digest,
                              void* workspace, size_t workspace_bytes, void* stream);
size_t canon_state_hash_workspace_bytes(int64_t n_tensors, const int64_t* nbytes);

/* ------------------------------------------------------------------------------------------------ */
/* Attention kernels of the paper's int8 path (training-details paragraph on int8 computation: the flash
   forward's P.V quantised to int8 per block on the integer matrix cores; the flash backward accumulating
   the query gradient in 64-bit fixed point).  Layouts as inside the decoder block: P and dS bf16
   [batch][n_heads][seq][seq] (row = query); V and K bf16 [batch][n_kv_heads][seq][head_dim]; O and dQ
   [batch][seq][n_heads * head_dim], head h at columns h * head_dim.  Query head h reads key/value head
   h / (n_heads / n_kv_heads).  Query i sees keys j <= i, and j > i - window when window > 0; entries of P
   and dS outside that set are not read (taken as +0).

   canon_attn_pv_i8 (R17): blocks of 64 queries x 64 keys of P and 64 keys x head_dim of V each get the step
     RN(amax * RN(1/127)) (amax by bit pattern), codes clamp(rne(RN(x / step)), -128, 127); a P block times a
     V block is an exact int32 sum, dequantised as RN(RN(RN32(acc) * sP) * sV); O is the R1 sum of these
     terms over key blocks in ascending order.  Writes O as fp32 (o_f32) and/or bf16 (o_bf16), either may
     be NULL.  head_dim a multiple of 32 up to 256; seq <= 8192.  workspace: device memory of
     canon_attn_pv_i8_workspace_bytes(batch, n_kv_heads, seq, head_dim) bytes, 256-byte aligned (the V codes
     and steps).
   canon_attn_dq_fixed (R18): dQ[i][c] = the sum over visible keys j of fx(dS[i][j] * K[j][c]), where fx(p)
     is the integer nearest to p * 2^frac_bits (ties to even), summed modulo 2^64 (the result is the same
     for every order of the keys), then times 2^-frac_bits rounded once to fp32 under R0.  frac_bits in
     [1, 62]; head_dim in {16, 32, 64, 128}. */
size_t canon_attn_pv_i8_workspace_bytes(int64_t batch, int64_t n_kv_heads, int64_t seq, int64_t head_dim);
canon_status canon_attn_pv_i8(int64_t batch, int64_t n_heads, int64_t n_kv_heads, int64_t seq, int64_t head_dim,
                              int64_t window, const uint16_t* P, const uint16_t* V, float* o_f32, uint16_t* o_bf16,
                              void* workspace, size_t workspace_bytes, void* stream);
canon_status canon_attn_dq_fixed(int64_t batch, int64_t n_heads, int64_t n_kv_heads, int64_t seq, int64_t head_dim,
                                 int64_t window, int32_t frac_bits, const uint16_t* dS, const uint16_t* K, float* dQ,
                                 void* stream);

/* LSQ gradient of a learned per-tensor activation step (R19; the int8 projections of canon_step with
   int8_linear): x bf16 [T, K] (the quantised activation), s: device fp32 scalar (the step), dx fp32 [T, K]
   (the gradient of the dequantised activation).  grad (device fp32 scalar) = RN(R1 over the flat index of
   RN(dx * delta) * RN32(1/sqrt(127 K))), delta = 0 if s is not > 0 once flushed or x/s is NaN, else with
   v = RN(x / s): -128 if v < -128, 127 if v > 127, RN(rne(v) - v) otherwise.  workspace: device memory of
   canon_lsq_step_grad_workspace_bytes(T, K) bytes (block sums). */
size_t canon_lsq_step_grad_workspace_bytes(int64_t T, int64_t K);
canon_status canon_lsq_step_grad(const canon_order* order, int64_t T, int64_t K, const uint16_t* x, const float* s,
                                 const float* dx, float* grad, void* workspace, size_t workspace_bytes, void* stream);

/* R11 embedding backward (the model section lists the embedding backward among the operators made bitwise
   reproducible): dE[v][:] = R1 over the ascending positions t with tokens[t] == v of dx[t][:] (plain terms:
   chains of 32 from +0, Algorithm 2 over the chain partials), for every v < V.  A row that never occurs is +0;
   a token outside [0, V) contributes nothing.  tokens: device int32 [T]; dx: device fp32 [T][d]; dE: device
   fp32 [V][d], fully written.  T < 2^25 (else CANON_EUNSUPPORTED).  workspace: device memory of
   canon_embed_bwd_workspace_bytes(T, d) bytes (sort keys, segment starts, chunk partials). */
size_t canon_embed_bwd_workspace_bytes(int64_t T, int64_t d);
canon_status canon_embed_bwd(const canon_order* order, int64_t T, int64_t V, int64_t d, const int32_t* tokens,
                             const float* dx, float* dE, void* workspace, size_t workspace_bytes, void* stream);

/* canon_lsq_step_grad without a workspace argument, for callers that cannot allocate device memory (code under
   HIP graph capture, serving loops, harnesses that forbid hipMalloc).  Same arguments, result and errors as
   canon_lsq_step_grad.  The block sums live in a 256 KiB device array inside the library, one copy per GPU,
   taken on the first call on that GPU and held until the process ends; no call allocates or frees memory.
   T * K may be at most canon_lsq_step_grad_noalloc_max_terms() (2^31); larger calls return
   CANON_EUNSUPPORTED and enqueue nothing.  Every call on one GPU shares its array: calls that overlap on one
   GPU (different streams, or host threads without ordering) race and give undefined results. */
canon_status canon_lsq_step_grad_noalloc(const canon_order* order, int64_t T, int64_t K, const uint16_t* x,
                                         const float* s, const float* dx, float* grad, void* stream);
int64_t canon_lsq_step_grad_noalloc_max_terms(void);

/* Device evaluation of the R0/R4 primitives, element by element, for testing the device math against
   the oracle: op 0 add, 1 sub, 2 mul, 3 fma(a,b,c), 4 div, 5 sqrt, 6 cexp, 7 clog, 8 sigmoid, 9 silu,
   10 bf16 round trip.  a, b, c, out: device fp32 [n] (b, c may be NULL when unused). */
canon_status canon_devmath(int32_t op, int64_t n, const float* a, const float* b, const float* c, float* out,
                           void* stream);

const char* canon_status_str(canon_status s);
int32_t canon_version(void);

#ifdef __cplusplus
}
#endif
#endif
