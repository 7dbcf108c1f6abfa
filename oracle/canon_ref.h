/*
 * canon_ref.h - CPU oracle of the canonical-order training step (CANON-v1).
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load this library.  It shares no code with
 * the GPU library: its own primitives, its own constants, its own header.
 *
 * All pointers are host memory owned by the caller.  bf16 tensors are passed as
 * uint16_t bit patterns.  Functions return 0 on success and a negative value on
 * invalid arguments.
 */
#ifndef CANON_REF_H
#define CANON_REF_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Model shape and the R16 variants (all zero: the plain block).  n_kv_heads: 0 (= n_heads) or a divisor
   of n_heads; qk_norm, embed_norm: 0 or 1; swa_window: 0 (full causal) or the window of the windowed
   layers, which are all but every swa_full_every-th and the last; z_loss: weight, 0 for none.
   pv_int8: 0 or 1, the attention forward's P.V by R17; dq_fixed_bits: 0 (dQ by R2) or F in [1, 62], the
   attention backward's dQ by R18 with F fractional bits.  int8_linear: 0 or 1, the four projections of every
   block in int8 (R19); each layer then has four more tensors after w_down, the bf16 activation steps
   sx_qkv, sx_o, sx_gate_up, sx_down (one element each, no weight decay). */
typedef struct {
  int32_t n_layers, d_model, n_heads, head_dim, d_ffn, vocab, seq, micro_seqs;
  float rms_eps;
  int32_t n_kv_heads, qk_norm, embed_norm, swa_window, swa_full_every;
  float z_loss;
  int32_t pv_int8, dq_fixed_bits;
  int32_t int8_linear;
} cref_model_cfg;

typedef struct {
  int32_t accum, dp_shard, dp_replicate;
} cref_plan;

typedef struct {
  float lr, beta1, one_minus_beta1, beta2, one_minus_beta2, inv_bc1, inv_bc2, eps, decay_factor;
} cref_adamw_consts;

/* R15 clip settings: max_norm > 0 (the clip threshold), spike_norm (a pre-clip norm not <= it is a
   spike), skip_steps >= 0 (updates skipped per spike, the spiking step included; 0: no spike rule). */
typedef struct {
  float max_norm, spike_norm;
  int32_t skip_steps;
} cref_clip_cfg;

/* ---- R0 primitives (scalar and vector forms, for the pins) ---- */
float cref_add(float a, float b);
float cref_sub(float a, float b);
float cref_mul(float a, float b);
float cref_fma(float a, float b, float c);
float cref_div(float a, float b);
float cref_sqrt(float a);
float cref_exp(float x);
float cref_log(float x);
float cref_sigmoid(float x);
float cref_silu(float x);
uint16_t cref_bf16(float x);
/* op: 0 add, 1 sub, 2 mul, 3 fma(a,b,c), 4 div, 5 sqrt, 6 exp, 7 log, 8 sigmoid, 9 silu, 10 bf16 round-trip */
int cref_prim(int32_t op, int64_t n, const float* a, const float* b, const float* c, float* out);

/* ---- R1 canonical reductions ---- */
float cref_rsum(const float* t, int64_t n, int64_t stride, int32_t chunk);
float cref_rdot_bf16(const uint16_t* a, int64_t sa, const uint16_t* b, int64_t sb, int64_t n, int32_t chunk);
float cref_rdot_f32(const float* a, int64_t sa, const float* b, int64_t sb, int64_t n, int32_t chunk);
/* Alg. 2 over nparts vectors of length len (parts[p*len ...]); *max_entries gets the deepest stack
   size seen, counting the incoming partial. */
int cref_treefold(const float* parts, int64_t nparts, int64_t len, float* out, int32_t* max_entries);

/* ---- R2 GEMM: C[i,j] = rsum_k A(i,k) B(k,j), bf16 operands, fp32 result ---- */
int cref_gemm(int32_t trans_a, int32_t trans_b, int64_t m, int64_t n, int64_t k, const uint16_t* a, int64_t lda,
              const uint16_t* b, int64_t ldb, float* c, int64_t ldc);

/* ---- R3 RMSNorm ---- */
int cref_rownorm_fwd(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps, uint16_t* y,
                     float* rstd);
int cref_rownorm_bwd(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, const float* rstd,
                     const float* dy, float* dx, float* dgain);
/* R3 forward with the output kept in fp32: y = RN(RN(x * r) * g) */
int cref_rownorm_fwd_f32(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps, float* y,
                         float* rstd);

/* ---- R5 causal softmax of raw scores (scale applied inside), R6 cross-entropy ----
   softmax_window: query i sees keys i - window < j <= i (window 0: all j <= i).
   xent_z: R6 plus the z-loss of weight z_loss (0: plain R6). */
int cref_softmax_causal(int64_t batch, int64_t s, const float* raw, float scale, uint16_t* probs);
int cref_softmax_window(int64_t batch, int64_t s, const float* raw, float scale, int64_t window, uint16_t* probs);
int cref_xent(int64_t rows, int64_t vocab, const uint16_t* logits, const int32_t* targets, float inv_tokens,
              uint16_t* dlogits, float* row_loss, float* mean_loss);
int cref_xent_z(int64_t rows, int64_t vocab, const uint16_t* logits, const int32_t* targets, float inv_tokens,
                float z_loss, uint16_t* dlogits, float* row_loss, float* mean_loss);

/* ---- R7 gradient plan (Alg. 1 + Alg. 2) ---- */
int cref_grad_accum(const cref_plan* plan, int64_t n, const float* const* grads, float* out);

/* ---- R9 AdamW ---- */
int cref_adamw(int64_t n_tensors, const int64_t* sizes, uint16_t* const* params, float* const* m, float* const* v,
               const float* const* grads, const uint8_t* decay_mask, const cref_adamw_consts* k);

/* ---- R15 global gradient norm, clip, spike skip ----
   global_norm: CRsqrt of the R1 sum of RN(g*g) over the tensors laid end to end in the given order.
   clip_decide: coef = CRdiv(max_norm, RN(norm + RN32(1e-6))); a norm that is not <= spike_norm sets
     *skip_state (updates still to skip) to skip_steps; *skipped = (*skip_state > 0), and a skipped step
     takes one off the counter.  skip_state may be NULL when skip_steps = 0.
   clip_apply: g <- RN(g * coef) in place when coef < 1. */
float cref_global_norm(int64_t n_tensors, const int64_t* sizes, const float* const* grads);
int cref_clip_decide(float norm, const cref_clip_cfg* k, int32_t* skip_state, float* coef, int32_t* skipped);
int cref_clip_apply(int64_t n_tensors, const int64_t* sizes, float* const* grads, float coef);

/* ---- one decoder block, forward + backward ----
   x, dy: fp32 [batch*seq, d]; w: the six block tensors in order attn_norm, w_qkv ([(H + 2 Hkv) hd, d]:
   query heads, key heads, value heads), w_o, ffn_norm, w_gate_up, w_down; y: block output; dx: input
   gradient; dw: six fp32 gradient buffers.  The block's attention window is cfg->swa_window. */
int cref_block_fwd_bwd(const cref_model_cfg* cfg, int32_t batch, const float* x, const float* dy,
                       const uint16_t* const* w, const float* rope_cos, const float* rope_sin, float* y, float* dx,
                       float* const* dw);

/* ---- full step: Alg. 1 over virtual ranks, then AdamW ----
   params/m/v: n_tensors = 3 + 6*n_layers (+1 with embed_norm) tensors in declared order (embed,
   [embed_norm], per layer: attn_norm, w_qkv, w_o, ffn_norm, w_gate_up, w_down; final_norm, head).  windows: [M][seq+1] int32 with
   M = dp_shard*dp_replicate*accum*micro_seqs.  grads_out (optional, may be NULL): per-tensor fp32
   buffers receiving the reduced gradient g (before any clip).  clip (optional): R15 between the
   plan and AdamW; norm_out gets the pre-clip norm, skip_state is the spike counter (in/out), and
   skipped_out (optional) is set to 1 when the update was skipped. */
int cref_step(const cref_model_cfg* cfg, const cref_plan* plan, uint16_t* const* params, float* const* m,
              float* const* v, const int32_t* windows, const float* rope_cos, const float* rope_sin,
              const cref_adamw_consts* k, const cref_clip_cfg* clip, float* loss_out, float* const* grads_out,
              float* norm_out, int32_t* skip_state, int32_t* skipped_out);

/* ---- R13 int8 quantised linear, forward (the W8A8 training path) ----
   quant_scales: per-row LSQ step of a bf16 matrix [rows][cols] re-pinned from the weights:
     s[r] = RN(RN(2 * RN(R1(|w[r,:]|) * RN(1/cols))) * RN(1/sqrt(127))).
   quantize: q = clamp(rne(RN(x / s)), -128, 127) for x fp32 (dtype 0) or bf16 (dtype 1), with one step
     per row (per_row = 1) or one for the whole tensor (per_row = 0); a step that is not > 0 after the
     input flush quantises to 0, and so does a NaN quotient.
   gemm_i8: acc[i][j] = sum_k a[i][k] * b[j][k] exactly (int8 operands, a [m][k], b [n][k]); acc (int32,
     optional) and y[i][j] = RN(RN(RN32(acc) * sa) * sb[j]) (fp32, optional), ldc for both.  k <= 65536. */
int cref_quant_scales(int64_t rows, int64_t cols, const uint16_t* w, float* scale);
int cref_quantize(int64_t rows, int64_t cols, int32_t dtype, const void* x, const float* scale, int32_t per_row,
                  int8_t* q);
int cref_gemm_i8(int64_t m, int64_t n, int64_t k, const int8_t* a, int64_t lda, const int8_t* b, int64_t ldb,
                 int32_t* acc, float* y, int64_t ldc, float sa, const float* sb);

/* ---- R14 int8 quantised linear, backward (straight-through estimator, Walsh-Hadamard rotated) ----
   fwht256: v (n values, n a multiple of 256) rotated in place block by block: per block of 256,
     butterflies (a, b) -> (RN(a + b), RN(a - b)) over strides 1, 2, ..., 128, then RN(x * 1/16).
   qlinear_bwd: given dy fp32 [T][N], the forward's int8 codes qx [T][K] (step sx) and qw [N][K] (steps
     sw[N]), computes dx = dy . W^ and dw = dy^T . X^ (W^ = RN(sw[n] qw), X^ = RN(sx qx)) as int8 GEMMs:
     each operand is rotated along the contraction dimension (N for dx, T for dw; a multiple of 256 when that output is asked for),
     quantised with the per-tensor step RN(amax * RN(1/127)) (amax: the largest |value|, NaN above all),
     multiplied exactly, and dequantised as RN(RN(RN32(acc) * s_left) * s_right).  dx or dw may be NULL. */
int cref_fwht256(int64_t n, float* v);
int cref_qlinear_bwd(int64_t T, int64_t N, int64_t K, const float* dy, const int8_t* qx, float sx, const int8_t* qw,
                     const float* sw, float* dx, float* dw);

/* ---- R17 int8 P.V inside the attention forward, one head ----
   P: bf16 [S][S] attention weights (masked entries +0), V: bf16 [S][hd]; O: fp32 [S][hd].  Blocks of 64
   queries x 64 keys of P and 64 keys x hd of V each get the step RN(amax * RN(1/127)) (amax by bit
   pattern); codes by R13's quantiser; each block product is an exact integer sum dequantised as
   RN(RN(RN32(acc) * sP) * sV); O = R1 over key blocks ascending. */
int cref_attn_pv_i8(int64_t S, int64_t hd, const uint16_t* P, const uint16_t* V, float* O);

/* ---- R18 dQ in 64-bit fixed point, one head ----
   dQ[i][c] = RN(sum_j fx(dS[i][j] * K[j][c]) * 2^-F) over the keys j the query sees (j <= i, and
   j > i - window when window > 0); fx(p) = the nearest integer to p * 2^F (ties to even), reduced modulo
   2^64; the sum wraps modulo 2^64 (two's complement), so its value does not depend on the order of the
   keys; the final rounding follows R0 (flush below 2^-126).  dS, K: bf16 [S][S], [S][hd]; dQ fp32. */
int cref_attn_dq_fixed(int64_t S, int64_t hd, int64_t window, int32_t frac_bits, const uint16_t* dS,
                       const uint16_t* K, float* dQ);
/* fx of one product, and the conversion of a wrapped sum back to fp32 (exported for the pins) */
uint64_t cref_fx_product(uint16_t a, uint16_t b, int32_t frac_bits);
float cref_fx_to_f32(uint64_t sum, int32_t frac_bits);

/* ---- R19 LSQ gradient of a per-tensor activation step ----
   x: bf16 [T][K] (the quantised activation), s: its step, dx: fp32 [T][K] (the gradient of the dequantised
   activation).  delta = 0 if s is not > 0 (after the input flush) or x/s is NaN; else with v = RN(x/s):
   -128 if v < -128, 127 if v > 127, RN(rne(v) - v) otherwise.  Returns RN(R1 over the flat index of
   RN(dx * delta) * RN32(1/sqrt(127 K))). */
float cref_lsq_step_grad(int64_t T, int64_t K, const uint16_t* x, float s, const float* dx);

/* R11 embedding backward: dE [V][d] from dx [T][d] and the tokens [T] of the microbatch (position t's token) */
int cref_embed_bwd(int64_t T, int64_t V, int64_t d, const int32_t* tok, const float* dx, float* dE);
/* SwiGLU per element (R4): a = bf16 forward output (if a), dg, du = bf16 gradients of g and u from the fp32
   gradient da of a (if da, dg and du) */
int cref_swiglu(int64_t n, const float* g, const float* u, const float* da, uint16_t* a, uint16_t* dg,
                uint16_t* du);
/* RN32(1/sqrt(n)) for 1 <= n < 2^60 (NaN otherwise), decided exactly */
float cref_inv_sqrt_int(int64_t n);
int cref_num_threads(void);
/* threads of the parallel loops (each parallel loop runs over independent outputs) */
void cref_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
