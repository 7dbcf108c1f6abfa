// canon_internal.h - argument structs and kernel launchers shared by the library's sources.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace canon {

enum { KMODE_FULL = 0, KMODE_TRAIL = 1, KMODE_LEAD = 2 };

// Reach of the causally skipping attention products (KMODE_TRAIL with the window kwin, KMODE_LEAD with kwin
// per K segment): with output tiles of at most 128 rows and chunks of 32, they read row i of a square
// per-head matrix (P, dS) only at columns i - kwin - kAttnLead <= j < floor(i / 128) * 128 + 128 (from j = 0
// without a window).  Writers of P and dS may leave everything outside that band unwritten.
constexpr int64_t kAttnLead = 157;

// One (possibly batched) GEMM.  Matrix z of the batch is (z1, z2) = (z / nb2, z % nb2), with operand
// offsets z1*s?1 + z2*s?2 (elements).
struct GemmArgs {
  const uint16_t* a;
  const uint16_t* b;
  void* c;
  int64_t m, n, k, lda, ldb, ldc;
  int64_t sa1, sa2, sb1, sb2, sc1, sc2;
  int64_t nb2, batch;
  int32_t trans_a, trans_b, out_bf16, kmode, tri_lower;
  int32_t vec;      // set by the launcher: 16-byte operand loads allowed
  int32_t b_group;  // > 1: B's inner batch offset is (z2 / b_group) * sb2 (grouped key/value heads)
  int64_t kwin;     // > 0: sliding attention window for the KMODE ranges and the tri_lower band
  int32_t zero_dead;  // EPI_DS with tri_lower: write the +0 of every tile without a visible entry (0: only
                      // of those left of the window band that the band's readers reach, see kAttnLead)
  int64_t kseg;       // > 0 (a multiple of 128 dividing k): the KMODE ranges repeat in every K segment of kseg
                      // (grouped heads stacked along K); 0: one segment
  // EPI_DS epilogue (attention backward, R5): the finished value d = dP[i][j] of a square per-head matrix
  // becomes dS[i][j] = bf16(RN(RN(P[i][j] * RN(d - D[i])) * ds_scale)) for j <= i (and j > i - ds_window
  // when ds_window > 0), +0 elsewhere, written as bf16 into C.  P: bf16 with leading dim ds_ldp and batch offsets ds_sp1/ds_sp2; D: fp32
  // per row with batch offsets ds_sd1/ds_sd2.
  int32_t epi;
  const uint16_t* ds_p;
  const float* ds_d;
  float ds_scale;
  int64_t ds_ldp, ds_sp1, ds_sp2, ds_sd1, ds_sd2;
  int64_t ds_window;
  float epi_scale;  // EPI_ACCUM
  const float* res;  // EPI_RES: fp32 [m][ldres] with C's batch offsets
  int64_t ldres;
};
// EPI_ACCUM: C = RN(C + RN(d * epi_scale)) (fp32 C); EPI_RES: C = RN(res + d) (fp32 C, the residual addition)
enum { EPI_NONE = 0, EPI_DS = 1, EPI_ACCUM = 2, EPI_RES = 3 };

hipError_t gemm_launch(const GemmArgs& g, hipStream_t s);

// gemm_i8.hip: exact int8 GEMM (a [m][k], b [n][k]) with optional int32 and dequantised fp32 outputs
struct GemmI8Args {
  const int8_t* a;
  const int8_t* b;
  int32_t* acc;     // may be null
  float* y;         // may be null
  const float* sa;  // device scalar (needed when y is set)
  const float* sb;  // device [n] (needed when y is set)
  int64_t m, n, k, lda, ldb, ldc;
  int32_t sb_scalar;  // 1: sb[0] for every column
  int32_t vec;        // set by the launcher
};
hipError_t gemm_i8_launch(const GemmI8Args& g, hipStream_t s);

// hash.hip: canonical state hash
struct HashTensor {
  const void* ptr;
  int64_t nbytes, leaves, leaf_offset;
  int32_t aligned;  // 16-byte aligned base: vector loads
};
int64_t hash_leaf_count(int64_t nbytes);
hipError_t hash_launch(int64_t n_tensors, const HashTensor* tens_dev, int64_t n_wg, const int32_t* wg_tensor,
                       const int64_t* wg_first, uint32_t* leaf_a, uint32_t* leaf_b, uint32_t* tensor_digests,
                       uint8_t* out, hipStream_t s);

// qlinear.hip: int8 backward (rotated straight-through gradients); dy fp32, or bf16 when dy_bf16
size_t qlinear_bwd_workspace_bytes(int64_t T, int64_t N, int64_t K);
hipError_t qlinear_bwd_launch(int64_t T, int64_t N, int64_t K, const void* dy, int dy_bf16, const int8_t* qx,
                              const float* sx, const int8_t* qw, const float* sw, float* dx, float* dw, void* ws,
                              hipStream_t s);
int gemm_max_levels();

// norm.hip: global gradient norm, clip coefficient, spike decision (R15)
struct NormSrc {
  const float* one;          // the whole vector in one buffer, or null
  const float* const* ptr;   // device [nt]: tensor bases (when one is null)
  const int64_t* start;      // device [nt + 1]: flat index of each tensor's first element; start[nt] = n
  int32_t nt;
};
struct ClipDecision {
  float max_norm, spike_norm;
  int32_t skip_steps;
  const int32_t* bad;    // may be null: a set flag marks the gradient invalid
  float* norm_out;       // may be null
  float* coef_out;       // device scalar, required
  int32_t* skip_state;   // may be null when skip_steps = 0
  int32_t* skip_flag;    // may be null: 1 when no update is to be applied
  int32_t* skipped_out;  // may be null
};
int64_t gnorm_blocks(int64_t n);  // block partials the launch needs
hipError_t gnorm_launch(const NormSrc& src, int64_t n, int vec4, float* part, const ClipDecision& d, hipStream_t s);
// g <- RN(g * *coef) when *coef < 1
hipError_t clip_scale_launch(int64_t n, float* g, const float* coef, hipStream_t s);

// rows.hip
hipError_t rownorm_fwd_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps,
                              uint16_t* y, float* rstd, hipStream_t s);
// the same with y kept fp32 (the embedding norm)
hipError_t rownorm_fwd_f32_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps,
                                  float* y, float* rstd, hipStream_t s);
// res (optional): dx = RN(res + the norm's gradient), the residual addition fused; dxb (optional): bf16 copy of dx
hipError_t rownorm_bwd_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, const float* rstd,
                              const float* dy, float* dx, float* dgain, hipStream_t s, const float* res = nullptr,
                              uint16_t* dxb = nullptr);
// window > 0: query i sees keys i - window < j <= i.  band = 0: every column of probs is written (+0 where
// masked); band = 1: only the columns the causally skipping products read (kAttnLead), the rest unwritten.
hipError_t softmax_causal_launch(int64_t rows, int64_t cols, const float* raw, float scale, int64_t window,
                                 uint16_t* probs, hipStream_t s, int band = 0);
hipError_t xent_launch(int64_t rows, int64_t vocab, const uint16_t* logits, const int32_t* targets,
                       float inv_tokens, float z_loss, uint16_t* dlogits, float* row_loss, float* mean_loss,
                       hipStream_t s);
hipError_t quant_scales_launch(int64_t rows, int64_t cols, const uint16_t* w, float* scale, hipStream_t s);
hipError_t attn_rowdot_launch(int64_t B, int64_t H, int64_t S, int64_t hd, const uint16_t* dO, const uint16_t* O,
                              int64_t ld, float* D, hipStream_t s);

// elementwise.hip
// qkv [T][(H + 2 Hkv) hd] -> q [B][H][S][hd], k and v [B][Hkv][S][hd] (bf16); with qk_norm, the gain-free
// per-head RMSNorm first, its r per head row into rq [T][H + Hkv]
hipError_t rope_qkv_launch(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd, const float* qkv,
                           const float* cosT, const float* sinT, int qk_norm, float eps, uint16_t* q, uint16_t* k,
                           uint16_t* v, float* rq, hipStream_t s);
// dq [T][H hd], dk [T][Hkv hd] -> the q and k columns of dqkv [T][(H + 2 Hkv) hd] (bf16); with qk_norm also
// the norm's backward (qkv: the forward's projection output, rq its r)
hipError_t rope_bwd_launch(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd, const float* dq, const float* dk,
                           const float* cosT, const float* sinT, int qk_norm, const float* qkv, const float* rq,
                           uint16_t* dqkv, hipStream_t s);
// [T][H hd] bf16 -> [B][H][S][hd]
hipError_t heads_major_launch(int64_t B, int64_t S, int64_t H, int64_t hd, const uint16_t* src, uint16_t* dst,
                              hipStream_t s);
hipError_t swiglu_fwd_launch(int64_t T, int64_t F, const float* gu, uint16_t* a, hipStream_t s);
hipError_t swiglu_bwd_launch(int64_t T, int64_t F, const float* gu, const float* da, uint16_t* dgu, hipStream_t s);
hipError_t add_f32_launch(int64_t n, const float* a, const float* b, float* out, hipStream_t s);
hipError_t cast_bf16_launch(int64_t n, const float* x, uint16_t* y, hipStream_t s);
hipError_t widen_bf16_launch(int64_t n, const uint16_t* x, float* y, hipStream_t s);
hipError_t token_check_launch(int64_t n, const int32_t* tok, int32_t bound, int32_t* bad_flag, hipStream_t s);
hipError_t embed_gather_launch(int64_t B, int64_t S, int64_t d, const int32_t* win, int64_t win_ld,
                               const uint16_t* E, int64_t V, float* x, hipStream_t s);
hipError_t labels_launch(int64_t B, int64_t S, const int32_t* win, int64_t win_ld, int32_t* lab, hipStream_t s);
// R11 embedding backward over T = B S positions (T < 2^25): dE [V][d] fully written; scratch of
// embed_bwd_scratch_bytes(T, d) bytes, 256-byte aligned
size_t embed_bwd_scratch_bytes(int64_t T, int64_t d);
hipError_t embed_bwd_launch(int64_t B, int64_t S, int64_t d, const int32_t* win, int64_t win_ld, int64_t V,
                            const float* dx, float* dE, void* scratch, hipStream_t s);
hipError_t quantize_launch(int64_t rows, int64_t cols, int32_t dtype, const void* x, const float* scale,
                           int32_t per_row, int8_t* q, hipStream_t s);
hipError_t devmath_launch(int32_t op, int64_t n, const float* a, const float* b, const float* c, float* out,
                          hipStream_t s);

// optim.hip
constexpr int kMaxFusedBuffers = 64;
struct PlanPtrs {
  const float* p[kMaxFusedBuffers];
};
hipError_t grad_accum_fused_launch(int accum, int dp_shard, int dp_replicate, int64_t n, const PlanPtrs& ptrs,
                                   float* out, hipStream_t s);
// out = (first ? +0 : out) + RN(grad * inv)        (Algorithm 1, microbatch accumulation)
hipError_t plan_accum_launch(int64_t n, const float* grad, float inv, int first, float* out, hipStream_t s);
// accum = 1: a rank's gradient into the ascending shard sum inner (first: shard 0), scaled by inv_shard on the
// last shard, in one pass
hipError_t plan_rank_launch(int64_t n, const float* grad, float inv_accum, int first, int last, float inv_shard,
                            float* inner, hipStream_t s);
// out = first ? a : RN(out + a)                      (ascending shard sum)
hipError_t plan_shard_launch(int64_t n, const float* a, int first, float* out, hipStream_t s);
// out = RN(lower + out)                              (fold merge, lower block on the left)
hipError_t plan_merge_launch(int64_t n, const float* lower, float* out, hipStream_t s);
// out = RN(x * inv) (in place allowed)
hipError_t plan_scale_launch(int64_t n, const float* x, float inv, float* out, hipStream_t s);
// gscale (may be null): the gradient is taken as RN(g * *gscale) when *gscale < 1 (the R15 clip)
hipError_t adamw_launch(int64_t n, uint16_t* p, float* m, float* v, const float* g, int decay, const float* consts9,
                        const float* gscale, const int32_t* skip_flag, hipStream_t s);
// R17 int8 P.V per block (attn_i8.hip): qvt int8 [B][Hkv][hd][64 nb] and sv fp32 [B][Hkv][nb] are scratch,
// nb = attn_pv_blocks(S); hd a multiple of 32 up to 256, S up to 8192.  R18 fixed-point dQ: hd in
// {16, 32, 64, 128}, F in [1, 62].
int64_t attn_pv_blocks(int64_t S);
hipError_t attn_pv_i8_launch(int64_t B, int64_t H, int64_t Hkv, int64_t S, int64_t hd, int64_t window,
                             const uint16_t* P, const uint16_t* V, float* of, uint16_t* ob, int64_t ldo, int8_t* qvt,
                             float* sv, hipStream_t s);
hipError_t attn_dq_fixed_launch(int64_t B, int64_t H, int64_t Hkv, int64_t S, int64_t hd, int64_t window, int F,
                                const uint16_t* dS, const uint16_t* K, float* dQ, int64_t ldq, hipStream_t s);
// lsq.hip: R19 gradient of a per-tensor activation step over n = T K terms (x bf16, dx fp32, step at s);
// part: scratch of lsq_grad_parts(n) floats; out: one float
int64_t lsq_grad_parts(int64_t n);
hipError_t lsq_grad_launch(int64_t n, const uint16_t* x, const float* s, const float* dx, float gamma, float* part,
                           float* out, hipStream_t st);
// the allocation-free variant: the calling GPU's copy of lsq.hip's device array of block sums (its address
// taken once per device), and the largest n it holds
hipError_t lsq_scratch(float** out);
int64_t lsq_noalloc_max_terms();
hipError_t set_nan_if_launch(const int32_t* flag, float* x, hipStream_t s);

}  // namespace canon
