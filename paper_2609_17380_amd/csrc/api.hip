// api.hip - the C ABI of libcanon: argument validation, workspace layout and the host-side orchestration
// of the decoder block and of the replayed step (Algorithm 1 over virtual ranks, then AdamW).
#include <hip/hip_runtime.h>
#include <math.h>
#include <string.h>

#include <vector>

#include "canon.h"
#include "canon_internal.h"

using namespace canon;

namespace {

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

canon_status check_order(const canon_order* o) {
  if (!o) return CANON_EINVAL;
  if (o->version != 1 || o->chunk != 32 || o->tree != CANON_TREE_BINARY_CARRY || o->ftz != 1)
    return CANON_EUNSUPPORTED;
  return CANON_OK;
}

canon_status dev(hipError_t e) { return e == hipSuccess ? CANON_OK : CANON_EDEVICE; }

#define TRY(expr)                                  \
  do {                                             \
    hipError_t _e = (expr);                        \
    if (_e != hipSuccess) return CANON_EDEVICE;    \
  } while (0)

GemmArgs mk(int ta, int tb, int64_t m, int64_t n, int64_t k, const uint16_t* a, int64_t lda, const uint16_t* b,
            int64_t ldb, void* c, int64_t ldc, int out_bf16 = 0) {
  GemmArgs g;
  memset(&g, 0, sizeof(g));
  g.a = a; g.b = b; g.c = c;
  g.m = m; g.n = n; g.k = k; g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  g.nb2 = 1; g.batch = 1;
  g.trans_a = ta; g.trans_b = tb; g.out_bf16 = out_bf16;
  g.kmode = KMODE_FULL; g.tri_lower = 0;
  return g;
}

// K limit of the register fold (chunk count must stay below 2^levels)
bool gemm_k_supported(int64_t k) { return ((k + 31) / 32) < (int64_t(1) << gemm_max_levels()); }

// Bump allocator over the caller's workspace (base == nullptr: size query only).
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base((char*)b) {}
  template <class T>
  T* take(int64_t n) {
    off = (off + 255) & ~size_t(255);
    T* p = base ? (T*)(base + off) : nullptr;
    off += sizeof(T) * (size_t)(n > 0 ? n : 1);
    return p;
  }
};

struct Dims {
  int64_t B, S, T, d, H, hd, F, V;
  int64_t Hkv, G, kvw, N;  // key/value heads, query heads per group, key width Hkv*hd, fused projection width
  int64_t window;          // this block's attention window (0: full causal)
  int qk_norm;
  int pv_int8, dq_bits;    // R17 int8 P.V; R18 fixed-point dQ with dq_bits fractional bits (0: off)
  int int8;                // R19: the four projections in int8
  float eps, scale, z_loss;
};

// floor(sqrt(x)) for x < 2^62: a binary64 estimate corrected in integers
uint64_t isqrt_u64(uint64_t x) {
  uint64_t r = (uint64_t)sqrt((double)x);
  while (r > 0 && r * r > x) --r;
  while ((r + 1) * (r + 1) <= x) ++r;
  return r;
}

// RN32(1/sqrt(n)) for 1 <= n < 2^40, in integers: with s such that 2^23 <= m = 2^s / sqrt(n) < 2^24, the
// significand is m rounded to an integer.  t = floor(2m) = floor(sqrt(floor(4^(s+1) / n))), and m rounds to
// (t + 1) / 2: 2m is never an odd integer (4^(s+1) / n would be an odd square), so no tie arises.
float rn32_inv_sqrt(int64_t n) {
  if (n < 1 || n >= ((int64_t)1 << 40)) return NAN;
  int bits = 0;
  while ((n >> bits) > 0) ++bits;
  int s = 23 + (bits + 1) / 2;
  uint64_t t = 0;
  for (;;) {
    const unsigned __int128 num = (unsigned __int128)1 << (2 * s + 2);
    t = isqrt_u64((uint64_t)(num / (unsigned __int128)n));
    if (t < ((uint64_t)1 << 24)) { ++s; continue; }   // m < 2^23
    if (t >= ((uint64_t)1 << 25)) { --s; continue; }  // m >= 2^24
    break;
  }
  uint64_t m = (t + 1) >> 1;
  if (m == ((uint64_t)1 << 24)) { m >>= 1; --s; }
  return ldexpf((float)m, -s);
}

float attn_scale(int64_t hd) { return rn32_inv_sqrt(hd); }  // 0x3DB504F3 for head_dim 128

int64_t kv_heads(const canon_model_cfg* c) { return c->n_kv_heads > 0 ? c->n_kv_heads : c->n_heads; }

// the attention window of layer l: the hybrid rule keeps every swa_full_every-th layer and the last full
int64_t layer_window(const canon_model_cfg* c, int64_t l) {
  if (c->swa_window == 0) return 0;
  if ((c->swa_full_every > 0 && (l + 1) % c->swa_full_every == 0) || l == c->n_layers - 1) return 0;
  return c->swa_window;
}

Dims dims_of(const canon_model_cfg* c, int64_t B) {
  Dims D;
  D.B = B; D.S = c->seq; D.T = B * c->seq; D.d = c->d_model; D.H = c->n_heads; D.hd = c->head_dim;
  D.F = c->d_ffn; D.V = c->vocab; D.eps = c->rms_eps; D.scale = attn_scale(c->head_dim);
  D.Hkv = kv_heads(c); D.G = D.H / D.Hkv; D.kvw = D.Hkv * D.hd; D.N = D.d + 2 * D.kvw;
  D.window = c->swa_window; D.qk_norm = c->qk_norm; D.z_loss = c->z_loss;
  D.pv_int8 = c->pv_int8; D.dq_bits = c->dq_fixed_bits;
  D.int8 = c->int8_linear;
  return D;
}

bool cfg_ok(const canon_model_cfg* c) {
  if (!(c && c->n_layers >= 1 && c->d_model > 0 && c->n_heads > 0 && c->head_dim > 0 && (c->head_dim % 2) == 0 &&
        (int64_t)c->n_heads * c->head_dim == c->d_model && c->d_ffn > 0 && c->vocab > 0 && c->seq > 0 &&
        c->micro_seqs > 0 && c->vocab <= 131072 && c->d_model <= 32768 && c->seq <= 32768))
    return false;
  if (c->n_kv_heads < 0 || (c->n_kv_heads > 0 && c->n_heads % c->n_kv_heads != 0)) return false;
  if ((c->qk_norm != 0 && c->qk_norm != 1) || (c->embed_norm != 0 && c->embed_norm != 1)) return false;
  if (c->swa_window < 0 || c->swa_full_every < 0 || !(c->z_loss >= 0.0f) || isinf(c->z_loss)) return false;
  if ((c->pv_int8 != 0 && c->pv_int8 != 1) || c->dq_fixed_bits < 0 || c->dq_fixed_bits > 62) return false;
  if (c->int8_linear != 0 && c->int8_linear != 1) return false;
  const int64_t G = c->n_heads / kv_heads(c);
  return gemm_k_supported(c->vocab) && gemm_k_supported((int64_t)c->seq * c->micro_seqs) &&
         gemm_k_supported(2 * (int64_t)c->d_ffn) && gemm_k_supported(c->d_model + 2 * kv_heads(c) * c->head_dim) &&
         gemm_k_supported(G * (int64_t)c->seq);
}

// shapes the R17, R18 and R19 kernels are built for (T tokens per block call)
bool variants_supported(const canon_model_cfg* c, int64_t T) {
  if (c->pv_int8 && (c->head_dim % 32 != 0 || c->head_dim > 256 || c->seq > 8192)) return false;
  if (c->dq_fixed_bits && c->head_dim != 16 && c->head_dim != 32 && c->head_dim != 64 && c->head_dim != 128)
    return false;
  if (c->int8_linear) {  // whole rotation blocks along every contraction of the int8 backward; the GEMM's k bound
    const int64_t d = c->d_model, F = c->d_ffn, N = d + 2 * kv_heads(c) * (int64_t)c->head_dim;
    if (T % 256 || d % 256 || (2 * F) % 256 || N % 256) return false;
    if (T > 65536 || N > 65536 || 2 * F > 65536 || F > 32768 || d > 32768) return false;
  }
  return true;
}

// R19: the four projections of a block, (N, K) and the tensor index of the weight within the layer
struct Proj {
  int64_t N, K;
};
void projections(const Dims& D, Proj (&p)[4]) {
  p[0] = {D.N, D.d};      // w_qkv
  p[1] = {D.d, D.d};      // w_o
  p[2] = {2 * D.F, D.d};  // w_gate_up
  p[3] = {D.d, D.F};      // w_down
}
const int kProjWeight[4] = {1, 2, 4, 5};  // index of each projection's weight among the layer's tensors

// LSQ's gradient scale RN32(1/sqrt(127 K)), correctly rounded
float lsq_gamma(int64_t K) { return rn32_inv_sqrt(127 * K); }

// activations a block saves for its backward pass
struct LayerSave {
  uint16_t *xn, *q, *k, *v, *P, *O, *hn, *a;
  float *rstd1, *h, *rstd2, *gu;
  float *qkv, *rq;  // QK-norm only: the projection output and the r of each q and k head row
  // R19: activation codes of the four projections, their steps widened to fp32, and the weights' codes
  // and re-pinned steps (computed once per call from the layer's weights)
  int8_t* qx[4];
  float* sxf;
  int8_t* qw[4];
  float* sw[4];
};

void carve_save(Carver& cv, const Dims& D, LayerSave& s) {
  const int64_t T = D.T, d = D.d;
  s.xn = cv.take<uint16_t>(T * d);
  s.rstd1 = cv.take<float>(T);
  s.q = cv.take<uint16_t>(T * d);
  s.k = cv.take<uint16_t>(T * D.kvw);
  s.v = cv.take<uint16_t>(T * D.kvw);
  s.qkv = D.qk_norm ? cv.take<float>(T * D.N) : nullptr;
  s.rq = D.qk_norm ? cv.take<float>(T * (D.H + D.Hkv)) : nullptr;
  s.P = cv.take<uint16_t>(D.B * D.H * D.S * D.S);
  s.O = cv.take<uint16_t>(T * d);
  s.h = cv.take<float>(T * d);
  s.hn = cv.take<uint16_t>(T * d);
  s.rstd2 = cv.take<float>(T);
  s.gu = cv.take<float>(T * 2 * D.F);
  s.a = cv.take<uint16_t>(T * D.F);
  Proj pj[4];
  projections(D, pj);
  for (int i = 0; i < 4; ++i) {
    s.qx[i] = D.int8 ? cv.take<int8_t>(T * pj[i].K) : nullptr;
    s.qw[i] = D.int8 ? cv.take<int8_t>(pj[i].N * pj[i].K) : nullptr;
    s.sw[i] = D.int8 ? cv.take<float>(pj[i].N) : nullptr;
  }
  s.sxf = D.int8 ? cv.take<float>(4) : nullptr;
}

// transient buffers shared by all layers
struct Scratch {
  float *qkv, *scores, *tmp_d, *da, *dtmp, *dtmp2, *dh, *dq, *dk, *Dv;
  uint16_t *dy_b, *dgu, *dO, *dS, *dqkv, *dOh;
  int8_t* qvt;  // R17: V codes, transposed per key block
  float* sv;    // R17: V block steps
  void* qws;    // R19: workspace of the rotated int8 backward
  float* lsq_part;  // R19: block sums of the activation-step gradients
  float* dOf;   // R19: fp32 gradient of the attention output before its bf16 rounding
};

void carve_scratch(Carver& cv, const Dims& D, Scratch& s) {
  const int64_t T = D.T, d = D.d;
  s.qkv = cv.take<float>(T * D.N);
  s.scores = cv.take<float>(D.B * D.H * D.S * D.S);
  s.tmp_d = cv.take<float>(T * d);
  s.da = cv.take<float>(T * D.F);
  s.dtmp = cv.take<float>(T * d);
  s.dtmp2 = cv.take<float>(T * d);
  s.dh = cv.take<float>(T * d);
  s.dq = cv.take<float>(T * d);
  s.dk = cv.take<float>(T * D.kvw);
  s.Dv = cv.take<float>(D.B * D.H * D.S);
  s.dy_b = cv.take<uint16_t>(T * d);
  s.dgu = cv.take<uint16_t>(T * 2 * D.F);
  s.dO = cv.take<uint16_t>(T * d);
  s.dS = cv.take<uint16_t>(D.B * D.H * D.S * D.S);
  s.dqkv = cv.take<uint16_t>(T * D.N);
  s.dOh = D.G > 1 ? cv.take<uint16_t>(T * d) : nullptr;
  const int64_t nb = attn_pv_blocks(D.S);
  s.qvt = D.pv_int8 ? cv.take<int8_t>(D.B * D.Hkv * D.hd * nb * 64) : nullptr;
  s.sv = D.pv_int8 ? cv.take<float>(D.B * D.Hkv * nb) : nullptr;
  s.qws = nullptr; s.lsq_part = nullptr; s.dOf = nullptr;
  if (D.int8) {
    Proj pj[4];
    projections(D, pj);
    int64_t parts = 1;
    size_t wsb = 0;
    for (int i = 0; i < 4; ++i) {
      const size_t b = qlinear_bwd_workspace_bytes(T, pj[i].N, pj[i].K);
      wsb = b > wsb ? b : wsb;
      const int64_t np = lsq_grad_parts(T * pj[i].K);
      parts = np > parts ? np : parts;
    }
    s.qws = cv.take<char>((int64_t)wsb);
    s.lsq_part = cv.take<float>(parts);
    s.dOf = cv.take<float>(T * d);
  }
}

// R19: codes and re-pinned steps of the layer's four projection weights, and its activation steps in fp32
// (w[6 + i]: the bf16 activation step of projection i)
canon_status prep_int8_layer(const Dims& D, const uint16_t* const* w, LayerSave& sv, hipStream_t s) {
  Proj pj[4];
  projections(D, pj);
  for (int i = 0; i < 4; ++i) {
    const uint16_t* W = w[kProjWeight[i]];
    TRY(quant_scales_launch(pj[i].N, pj[i].K, W, sv.sw[i], s));
    TRY(quantize_launch(pj[i].N, pj[i].K, CANON_BF16, W, sv.sw[i], 1, sv.qw[i], s));
    TRY(widen_bf16_launch(1, w[6 + i], sv.sxf + i, s));
  }
  return CANON_OK;
}

// R19 forward of projection i: Y [T][N] from the bf16 input X [T][K]
canon_status qproj_fwd(const Dims& D, int i, const uint16_t* X, float* Y, LayerSave& sv, hipStream_t s) {
  Proj pj[4];
  projections(D, pj);
  const int64_t N = pj[i].N, K = pj[i].K;
  TRY(quantize_launch(D.T, K, CANON_BF16, X, sv.sxf + i, 0, sv.qx[i], s));
  GemmI8Args g{};
  g.a = sv.qx[i]; g.b = sv.qw[i]; g.y = Y; g.sa = sv.sxf + i; g.sb = sv.sw[i];
  g.m = D.T; g.n = N; g.k = K; g.lda = K; g.ldb = K; g.ldc = N;
  TRY(gemm_i8_launch(g, s));
  return CANON_OK;
}

// R19 backward of projection i: G16 the bf16 gradient of its output [T][N]; dX [T][K], dW [N][K] by the rotated
// int8 backward; dsx the activation step's gradient (X the bf16 input of the forward)
canon_status qproj_bwd(const Dims& D, int i, const uint16_t* G16, const uint16_t* X, float* dX, float* dW, float* dsx,
                       const LayerSave& sv, Scratch& sc, hipStream_t s) {
  Proj pj[4];
  projections(D, pj);
  const int64_t N = pj[i].N, K = pj[i].K;
  TRY(qlinear_bwd_launch(D.T, N, K, G16, 1, sv.qx[i], sv.sxf + i, sv.qw[i], sv.sw[i], dX, dW, sc.qws, s));
  TRY(lsq_grad_launch(D.T * K, X, sv.sxf + i, dX, lsq_gamma(K), sc.lsq_part, dsx, s));
  return CANON_OK;
}

hipError_t gemm(const GemmArgs& g, hipStream_t s) { return gemm_launch(g, s); }

// per-head batched GEMM over (b, h): A/B/C offsets b*s?1 + h*s?2
GemmArgs batched(GemmArgs g, const Dims& D, int64_t sa1, int64_t sa2, int64_t sb1, int64_t sb2, int64_t sc1,
                 int64_t sc2) {
  g.batch = D.B * D.H; g.nb2 = D.H;
  g.sa1 = sa1; g.sa2 = sa2; g.sb1 = sb1; g.sb2 = sb2; g.sc1 = sc1; g.sc2 = sc2;
  return g;
}

// Forward of one block: x (input, kept by the caller) -> y; activations saved in sv.  Query head h reads
// key/value head h / G (the GEMMs' b_group); with QK-norm the projection output is kept for the backward.
canon_status block_forward(const Dims& D, const uint16_t* const* w, const float* cosT, const float* sinT,
                           const float* x, LayerSave& sv, Scratch& sc, float* y, hipStream_t s) {
  const int64_t T = D.T, d = D.d, S = D.S, H = D.H, Hkv = D.Hkv, hd = D.hd, F = D.F, N = D.N;
  float* qkv = D.qk_norm ? sv.qkv : sc.qkv;
  TRY(rownorm_fwd_launch(T, d, x, w[0], D.eps, sv.xn, sv.rstd1, s));
  if (D.int8) {
    canon_status st = qproj_fwd(D, 0, sv.xn, qkv, sv, s);
    if (st != CANON_OK) return st;
  } else {
    TRY(gemm(mk(0, 1, T, N, d, sv.xn, d, w[1], d, qkv, N), s));
  }
  TRY(rope_qkv_launch(D.B, S, H, Hkv, hd, qkv, cosT, sinT, D.qk_norm, D.eps, sv.q, sv.k, sv.v, sv.rq, s));
  {  // raw scores Q K^T, lower-triangle tiles only
    GemmArgs g = batched(mk(0, 1, S, S, hd, sv.q, hd, sv.k, hd, sc.scores, S), D, H * S * hd, S * hd,
                         Hkv * S * hd, S * hd, H * S * S, S * S);
    g.tri_lower = 1;
    g.kwin = D.window;  // tiles left of the window band are not computed (the softmax reads none of them)
    g.b_group = (int32_t)D.G;
    TRY(gemm(g, s));
  }
  // P is written only where the P.V and dV products read it, unless dV reads every query (grouped heads
  // with S not a multiple of 128: one contraction without per-head ranges)
  const int band = (D.G == 1 || S % 128 == 0) ? 1 : 0;
  TRY(softmax_causal_launch(D.B * H * S, S, sc.scores, D.scale, D.window, sv.P, s, band));
  if (D.pv_int8) {  // R17: O = P V on the int8 matrix cores, per block of 64 queries x 64 keys
    TRY(attn_pv_i8_launch(D.B, H, Hkv, S, hd, D.window, sv.P, sv.v, nullptr, sv.O, d, sc.qvt, sc.sv, s));
  } else {  // O = P V (keys beyond the tile's last query are masked chunks), bf16 into [T, d]
    GemmArgs g = batched(mk(0, 0, S, hd, S, sv.P, S, sv.v, hd, sv.O, d, 1), D, H * S * S, S * S, Hkv * S * hd,
                         S * hd, S * d, hd);
    g.kmode = KMODE_TRAIL;
    g.kwin = D.window;
    g.b_group = (int32_t)D.G;
    TRY(gemm(g, s));
  }
  if (D.int8) {
    canon_status st = qproj_fwd(D, 1, sv.O, sc.tmp_d, sv, s);
    if (st != CANON_OK) return st;
    TRY(add_f32_launch(T * d, x, sc.tmp_d, sv.h, s));
  } else {  // h = x + O W_o^T, the residual addition in the GEMM's epilogue
    GemmArgs g = mk(0, 1, T, d, d, sv.O, d, w[2], d, sv.h, d);
    g.epi = EPI_RES; g.res = x; g.ldres = d;
    TRY(gemm(g, s));
  }
  TRY(rownorm_fwd_launch(T, d, sv.h, w[3], D.eps, sv.hn, sv.rstd2, s));
  if (D.int8) {
    canon_status st = qproj_fwd(D, 2, sv.hn, sv.gu, sv, s);
    if (st != CANON_OK) return st;
  } else {
    TRY(gemm(mk(0, 1, T, 2 * F, d, sv.hn, d, w[4], d, sv.gu, 2 * F), s));
  }
  TRY(swiglu_fwd_launch(T, F, sv.gu, sv.a, s));
  if (D.int8) {
    canon_status st = qproj_fwd(D, 3, sv.a, sc.tmp_d, sv, s);
    if (st != CANON_OK) return st;
    TRY(add_f32_launch(T * d, sv.h, sc.tmp_d, y, s));
  } else {  // y = h + a W_down^T
    GemmArgs g = mk(0, 1, T, d, F, sv.a, F, w[5], F, y, d);
    g.epi = EPI_RES; g.res = sv.h; g.ldres = d;
    TRY(gemm(g, s));
  }
  return CANON_OK;
}

// Backward of one block: dy (gradient of the block output) -> dx; weight gradients into dw[0..5].  The
// gradient of a shared key (value) head is one contraction over its group's query heads and their queries,
// heads in order: the group's dS (P) and Q (dO) rows are contiguous head after head, one GEMM with K = G*S.
canon_status block_backward(const Dims& D, const uint16_t* const* w, const float* cosT, const float* sinT,
                            const float* x, const LayerSave& sv, Scratch& sc, const float* dy, float* dx,
                            float* const* dw, hipStream_t s) {
  const int64_t T = D.T, d = D.d, S = D.S, H = D.H, Hkv = D.Hkv, G = D.G, hd = D.hd, F = D.F, N = D.N;
  const int64_t kvw = D.kvw;
  canon_status qst = CANON_OK;
  TRY(cast_bf16_launch(T * d, dy, sc.dy_b, s));
  if (D.int8) {
    if ((qst = qproj_bwd(D, 3, sc.dy_b, sv.a, sc.da, dw[5], dw[9], sv, sc, s)) != CANON_OK) return qst;
  } else {
    TRY(gemm(mk(1, 0, d, F, T, sc.dy_b, d, sv.a, F, dw[5], F), s));        // dW_down = dy^T a
    TRY(gemm(mk(0, 0, T, F, d, sc.dy_b, d, w[5], F, sc.da, F), s));        // da = dy W_down
  }
  TRY(swiglu_bwd_launch(T, F, sv.gu, sc.da, sc.dgu, s));
  if (D.int8) {
    if ((qst = qproj_bwd(D, 2, sc.dgu, sv.hn, sc.dtmp, dw[4], dw[8], sv, sc, s)) != CANON_OK) return qst;
  } else {
    TRY(gemm(mk(1, 0, 2 * F, d, T, sc.dgu, 2 * F, sv.hn, d, dw[4], d), s)); // dW_gate_up = dgu^T hn
    TRY(gemm(mk(0, 0, T, d, 2 * F, sc.dgu, 2 * F, w[4], d, sc.dtmp, d), s)); // dhn = dgu W_gate_up
  }
  // dh = dy + norm path (the residual addition inside the norm's backward), and its bf16 copy
  TRY(rownorm_bwd_launch(T, d, sv.h, w[3], sv.rstd2, sc.dtmp, sc.dh, dw[3], s, dy, sc.dy_b));
  if (D.int8) {
    if ((qst = qproj_bwd(D, 1, sc.dy_b, sv.O, sc.dOf, dw[2], dw[7], sv, sc, s)) != CANON_OK) return qst;
    TRY(cast_bf16_launch(T * d, sc.dOf, sc.dO, s));
  } else {
    TRY(gemm(mk(1, 0, d, d, T, sc.dy_b, d, sv.O, d, dw[2], d), s));        // dW_o = dh^T O
    TRY(gemm(mk(0, 0, T, d, d, sc.dy_b, d, w[2], d, sc.dO, d, 1), s));     // dO = dh W_o (bf16)
  }
  TRY(attn_rowdot_launch(D.B, H, S, hd, sc.dO, sv.O, d, sc.Dv, s));      // D = rowsum(dO * O)
  {  // dP = dO V^T, turned into dS = P * (dP - D) * c in the epilogue (bf16).  Tiles with no visible entry are
     // not computed: those left of the window band that the windowed dQ and dK ranges reach get their +0
     // written, the rest stay unwritten; with grouped heads and S not a multiple of 128, dK reads each
     // head's dS whole, and every such tile gets its +0.
    GemmArgs g = batched(mk(0, 1, S, S, hd, sc.dO, d, sv.v, hd, sc.dS, S), D, S * d, hd, Hkv * S * hd, S * hd,
                         H * S * S, S * S);
    g.tri_lower = 1;
    g.kwin = D.window;
    g.zero_dead = (G > 1 && S % 128 != 0) ? 1 : 0;
    g.b_group = (int32_t)G;
    g.epi = EPI_DS;
    g.ds_p = sv.P; g.ds_d = sc.Dv; g.ds_scale = D.scale; g.ds_window = D.window;
    g.ds_ldp = S; g.ds_sp1 = H * S * S; g.ds_sp2 = S * S; g.ds_sd1 = H * S; g.ds_sd2 = S;
    TRY(gemm(g, s));
  }
  if (D.dq_bits) {  // R18: dQ = dS K accumulated in 64-bit fixed point
    TRY(attn_dq_fixed_launch(D.B, H, Hkv, S, hd, D.window, D.dq_bits, sc.dS, sv.k, sc.dq, d, s));
  } else {  // dQ = dS K (over keys)
    GemmArgs g = batched(mk(0, 0, S, hd, S, sc.dS, S, sv.k, hd, sc.dq, d), D, H * S * S, S * S, Hkv * S * hd,
                         S * hd, S * d, hd);
    g.kmode = KMODE_TRAIL;
    g.kwin = D.window;
    g.b_group = (int32_t)G;
    TRY(gemm(g, s));
  }
  // per (batch, key/value head): the group's G heads stacked along the contraction
  auto grouped = [&](GemmArgs g, int64_t sa1, int64_t sa2, int64_t sb1, int64_t sb2, int64_t sc1, int64_t sc2) {
    g.batch = D.B * Hkv; g.nb2 = Hkv;
    g.sa1 = sa1; g.sa2 = sa2; g.sb1 = sb1; g.sb2 = sb2; g.sc1 = sc1; g.sc2 = sc2;
    // in each head's segment of the contraction, queries before the key tile (and after its window) are
    // zero chunks; segments need S to be a multiple of 128 (whole groups of four chunks)
    const bool seg = G == 1 || S % 128 == 0;
    g.kmode = seg ? KMODE_LEAD : KMODE_FULL;
    if (seg) g.kwin = D.window;
    if (G > 1 && seg) g.kseg = S;
    return g;
  };
  // dK = sum over the group of dS^T Q (over the group's queries)
  TRY(gemm(grouped(mk(1, 0, S, hd, G * S, sc.dS, S, sv.q, hd, sc.dk, kvw), H * S * S, G * S * S, H * S * hd,
                   G * S * hd, S * kvw, hd), s));
  // dV = sum over the group of P^T dO, bf16 into the value columns of dqkv
  const uint16_t* dO_heads = sc.dO;
  int64_t dO_s1 = S * d, dO_s2 = hd, dO_ld = d;
  if (G > 1) {  // the group's dO rows must be contiguous: head-major copy
    TRY(heads_major_launch(D.B, S, H, hd, sc.dO, sc.dOh, s));
    dO_heads = sc.dOh; dO_s1 = H * S * hd; dO_s2 = G * S * hd; dO_ld = hd;
  }
  TRY(gemm(grouped(mk(1, 0, S, hd, G * S, sv.P, S, dO_heads, dO_ld, sc.dqkv + d + kvw, N, 1), H * S * S, G * S * S,
                   dO_s1, dO_s2, S * N, hd), s));
  TRY(rope_bwd_launch(D.B, S, H, Hkv, hd, sc.dq, sc.dk, cosT, sinT, D.qk_norm, sv.qkv, sv.rq, sc.dqkv, s));
  if (D.int8) {
    if ((qst = qproj_bwd(D, 0, sc.dqkv, sv.xn, sc.dtmp, dw[1], dw[6], sv, sc, s)) != CANON_OK) return qst;
  } else {
    TRY(gemm(mk(1, 0, N, d, T, sc.dqkv, N, sv.xn, d, dw[1], d), s));       // dW_qkv = dqkv^T xn
    TRY(gemm(mk(0, 0, T, d, N, sc.dqkv, N, w[1], d, sc.dtmp, d), s));      // dxn = dqkv W_qkv
  }
  TRY(rownorm_bwd_launch(T, d, x, w[0], sv.rstd1, sc.dtmp, dx, dw[0], s, sc.dh));  // dx = dh + norm path
  return CANON_OK;
}

// ---- step layout ---------------------------------------------------------------------------------
int bit_length(int64_t x) {
  int b = 0;
  while ((int64_t(1) << b) <= x) ++b;
  return b;
}

// tensors in the declared order: embed, [embed_norm], per layer attn_norm, w_qkv, w_o, ffn_norm, w_gate_up,
// w_down [, sx_qkv, sx_o, sx_gate_up, sx_down], then final_norm, head
void tensor_sizes(const canon_model_cfg* c, std::vector<int64_t>& sz, std::vector<uint8_t>& decay) {
  const int64_t d = c->d_model, F = c->d_ffn, V = c->vocab;
  const int64_t N = d + 2 * kv_heads(c) * c->head_dim;
  sz.clear(); decay.clear();
  sz.push_back(V * d); decay.push_back(0);
  if (c->embed_norm) { sz.push_back(d); decay.push_back(0); }
  for (int l = 0; l < c->n_layers; ++l) {
    int64_t s6[6] = {d, N * d, d * d, d, 2 * F * d, d * F};
    uint8_t d6[6] = {0, 1, 1, 0, 1, 1};
    for (int i = 0; i < 6; ++i) { sz.push_back(s6[i]); decay.push_back(d6[i]); }
    if (c->int8_linear)  // R19 activation steps of the four projections
      for (int i = 0; i < 4; ++i) { sz.push_back(1); decay.push_back(0); }
  }
  sz.push_back(d); decay.push_back(0);
  sz.push_back(V * d); decay.push_back(1);
}

// slots of the gradient plan (see the plan cursor below): 256-byte aligned, n floats each
int64_t plan_slot_stride(int64_t n) { return (n + 63) & ~int64_t(63); }  // 256-byte aligned slots
int plan_slot_count(const canon_dp_plan& p) { return (p.accum > 1 ? 1 : 0) + bit_length(p.dp_replicate) + 1; }
bool plan_ok(const canon_dp_plan* p) {
  return p && p->accum >= 1 && p->dp_shard >= 1 && p->dp_replicate >= 1 &&
         (int64_t)p->accum * p->dp_shard * p->dp_replicate <= INT32_MAX;
}
int64_t plan_total(const canon_dp_plan& p) { return (int64_t)p.accum * p.dp_shard * p.dp_replicate; }

struct StepLayout {
  std::vector<LayerSave> saves;
  std::vector<float*> xs;  // residual stream: xs[0] = embedding output, xs[l+1] = block l output
  Scratch sc;
  uint16_t *xf, *logits, *dlogits;
  float *rstdf, *row_loss, *dxf, *dxA, *dxB;
  int32_t *win, *lab, *bad;
  void* embed_scratch;
  float* grad;            // one microbatch's gradient, all tensors
  float* plan_slots;      // the gradient plan's slots (rank accumulator, shard sum, Algorithm 2 stack)
  float* loss_mb;         // [1]
  float* loss_slots;      // the same plan over the microbatch losses
  float* norm_part;       // R15 block sums
  float* clip_coef;       // [1]
  int32_t* skip;          // [1]: no update this step (bad token or spike window)
  float* x_emb;           // embedding norm: the gathered rows [T][d]
  float* rstd_emb;        // embedding norm: r per row [T]
  char* hash_ws;          // the per-step state hash's tables and leaf digests
};

// the tensors of the per-step state hash: the step's windows, then the parameters, m, v and the reduced
// gradient, each in the declared order
void step_hash_sizes(const canon_model_cfg* c, const canon_dp_plan* p, std::vector<int64_t>& nb) {
  std::vector<int64_t> sz;
  std::vector<uint8_t> decay;
  tensor_sizes(c, sz, decay);
  const int64_t M = (int64_t)p->accum * p->dp_shard * p->dp_replicate * c->micro_seqs;
  nb.clear();
  nb.push_back(M * (c->seq + 1) * (int64_t)sizeof(int32_t));
  for (int64_t x : sz) nb.push_back(2 * x);
  for (int rep = 0; rep < 3; ++rep)
    for (int64_t x : sz) nb.push_back(4 * x);
}
size_t step_hash_bytes(const canon_model_cfg* c, const canon_dp_plan* p);

void carve_step(Carver& cv, const canon_model_cfg* c, const canon_dp_plan* p, int64_t P, StepLayout& L) {
  Dims D = dims_of(c, c->micro_seqs);
  L.saves.resize(c->n_layers);
  for (auto& s : L.saves) carve_save(cv, D, s);
  L.xs.resize(c->n_layers + 1);
  for (auto& x : L.xs) x = cv.take<float>(D.T * D.d);
  carve_scratch(cv, D, L.sc);
  L.xf = cv.take<uint16_t>(D.T * D.d);
  L.rstdf = cv.take<float>(D.T);
  L.logits = cv.take<uint16_t>(D.T * D.V);
  L.dlogits = cv.take<uint16_t>(D.T * D.V);
  L.row_loss = cv.take<float>(D.T);
  L.dxf = cv.take<float>(D.T * D.d);
  L.dxA = cv.take<float>(D.T * D.d);
  L.dxB = cv.take<float>(D.T * D.d);
  L.win = cv.take<int32_t>((int64_t)c->micro_seqs * (c->seq + 1));
  L.lab = cv.take<int32_t>(D.T);
  L.bad = cv.take<int32_t>(1);
  L.embed_scratch = cv.take<char>((int64_t)embed_bwd_scratch_bytes(D.T, D.d));
  L.grad = cv.take<float>(P);
  L.plan_slots = cv.take<float>(plan_slot_stride(P) * plan_slot_count(*p));
  L.loss_mb = cv.take<float>(1);
  L.loss_slots = cv.take<float>(plan_slot_stride(1) * plan_slot_count(*p));
  L.norm_part = cv.take<float>(gnorm_blocks(P));
  L.clip_coef = cv.take<float>(1);
  L.skip = cv.take<int32_t>(1);
  L.x_emb = c->embed_norm ? cv.take<float>(D.T * D.d) : nullptr;
  L.rstd_emb = c->embed_norm ? cv.take<float>(D.T) : nullptr;
  L.hash_ws = cv.take<char>((int64_t)step_hash_bytes(c, p));
}

// Algorithm 1 driven from the host, one microbatch at a time, over device slots of n floats each (the
// gradient, or the loss with n = 1).  The position and the Algorithm 2 stack live in a plain host record
// (canon_plan_cursor) and the partial sums in the caller's slots, so the plan can stop after any microbatch,
// be persisted (record + slot bytes) and resume in other memory.  Slot 0 is the rank accumulator when
// accum > 1; the others hold the shard sum being built and the stack entries.
void plan_cursor_init(const canon_dp_plan& p, int64_t n, canon_plan_cursor* c) {
  memset(c, 0, sizeof(*c));
  c->plan = p;
  c->n = n;
  c->next = 0;
  c->inner = -1;
  c->depth = 0;
}

// The record must be one that plan_cursor_init and plan_cursor_push can produce: its stack shape and the
// presence of a shard sum follow from `next`, and the slots are distinct and in range.
bool plan_cursor_valid(const canon_plan_cursor* c) {
  if (!c || !plan_ok(&c->plan) || c->n < 0) return false;
  const canon_dp_plan& p = c->plan;
  const int64_t total = plan_total(p);
  if (c->next < 0 || c->next > total) return false;
  const int64_t r = c->next / p.accum;               // ranks whose microbatches are all in (== N at the end)
  const int64_t groups = r / p.dp_shard;             // replica groups complete
  const bool partial_group = (r % p.dp_shard) != 0;  // some shards of the current replica are in
  if (partial_group != (c->inner >= 0)) return false;
  int64_t bits = groups;
  int depth = 0;
  for (int L = 30; L >= 0; --L) {
    if (!((bits >> L) & 1)) continue;
    if (depth >= CANON_PLAN_MAX_DEPTH || c->level[depth] != L) return false;
    ++depth;
  }
  if (depth != c->depth) return false;
  const int first = p.accum > 1 ? 1 : 0, nslots = plan_slot_count(p);
  uint64_t used = 0;
  for (int i = 0; i <= depth; ++i) {
    const int sl = i < depth ? c->slot[i] : c->inner;
    if (i == depth && sl < 0) continue;
    if (sl < first || sl >= nslots || ((used >> sl) & 1)) return false;
    used |= uint64_t(1) << sl;
  }
  return true;
}

int plan_take_slot(const canon_plan_cursor* c) {
  const int first = c->plan.accum > 1 ? 1 : 0, nslots = plan_slot_count(c->plan);
  for (int sl = first; sl < nslots; ++sl) {
    bool busy = sl == c->inner;
    for (int i = 0; i < c->depth; ++i) busy = busy || c->slot[i] == sl;
    if (!busy) return sl;
  }
  return -1;  // cannot happen for a valid cursor
}

// microbatch k of rank r (r = next / accum, k = next % accum) produced `grad`
hipError_t plan_cursor_push(canon_plan_cursor* c, float* base, const float* grad, hipStream_t s) {
  const canon_dp_plan& p = c->plan;
  const int64_t n = c->n, st = plan_slot_stride(n);
  const int r = (int)(c->next / p.accum), k = (int)(c->next % p.accum);
  const int shard = r % p.dp_shard;
  const float inv_accum = (float)(1.0 / p.accum), inv_shard = (float)(1.0 / p.dp_shard);
  auto slot = [&](int i) { return base + st * i; };
  hipError_t e = hipSuccess;
  ++c->next;
  if (p.accum == 1) {  // one microbatch per rank: its sum, the shard sum and the last shard's scale in one pass
    if (shard == 0) c->inner = plan_take_slot(c);
    if (n > 0) e = plan_rank_launch(n, grad, inv_accum, shard == 0, shard == p.dp_shard - 1, inv_shard, slot(c->inner), s);
    if (e != hipSuccess || shard != p.dp_shard - 1) return e;
  } else {
    float* g_r = slot(0);
    if (n > 0) e = plan_accum_launch(n, grad, inv_accum, k == 0, g_r, s);
    if (e != hipSuccess || k != p.accum - 1) return e;
    if (shard == 0) c->inner = plan_take_slot(c);
    if (n > 0) e = plan_shard_launch(n, g_r, shard == 0, slot(c->inner), s);
    if (e != hipSuccess || shard != p.dp_shard - 1) return e;
    if (n > 0) e = plan_scale_launch(n, slot(c->inner), inv_shard, slot(c->inner), s);
  }
  // Algorithm 2: push the replica's average at level 0 and carry
  int level = 0, part = c->inner;
  while (e == hipSuccess && c->depth > 0 && c->level[c->depth - 1] == level) {
    const int lower = c->slot[c->depth - 1];
    if (n > 0) e = plan_merge_launch(n, slot(lower), slot(part), s);  // part = lower + part
    --c->depth;
    ++level;
  }
  c->level[c->depth] = level;
  c->slot[c->depth] = part;
  ++c->depth;
  c->inner = -1;
  return e;
}

// Result of Algorithm 2 (the entries from the top of the stack down, each added on the left) times
// 1/dp_replicate, left in a slot whose address is returned (the caller's `out` when given).
float* plan_cursor_finish(canon_plan_cursor* c, float* base, float* out, hipStream_t s, hipError_t* err) {
  const int64_t n = c->n, st = plan_slot_stride(n);
  float* acc = base + st * c->slot[c->depth - 1];
  hipError_t e = hipSuccess;
  for (int i = c->depth - 2; i >= 0 && e == hipSuccess; --i)
    if (n > 0) e = plan_merge_launch(n, base + st * c->slot[i], acc, s);
  const float inv_rep = (float)(1.0 / c->plan.dp_replicate);
  float* dst = out ? out : acc;
  // RN(x * 1) = x for every x the sums can hold (never subnormal): one replica needs no pass
  if (e == hipSuccess && n > 0) {
    if (inv_rep != 1.0f) e = plan_scale_launch(n, acc, inv_rep, dst, s);
    else if (dst != acc) e = hipMemcpyAsync(dst, acc, sizeof(float) * n, hipMemcpyDeviceToDevice, s);
  }
  *err = e;
  return dst;
}

struct HashPlan {
  int64_t total_leaves = 0, n_wg = 0;
  size_t off_tens = 0, off_wgt = 0, off_wgf = 0, off_la = 0, off_lb = 0, off_td = 0, bytes = 0;
};

HashPlan hash_plan(int64_t n, const int64_t* nbytes) {
  HashPlan hp;
  for (int64_t t = 0; t < n; ++t) {
    const int64_t w = hash_leaf_count(nbytes[t]);
    hp.total_leaves += w;
    hp.n_wg += (w + 255) / 256;
  }
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  size_t o = 0;
  hp.off_tens = o; o += up(sizeof(HashTensor) * (size_t)n);
  hp.off_wgt = o; o += up(sizeof(int32_t) * (size_t)hp.n_wg);
  hp.off_wgf = o; o += up(sizeof(int64_t) * (size_t)hp.n_wg);
  hp.off_la = o; o += up(32 * (size_t)hp.total_leaves);
  hp.off_lb = o; o += up(32 * (size_t)hp.total_leaves);
  hp.off_td = o; o += up(32 * (size_t)n);
  hp.bytes = o;
  return hp;
}

size_t step_hash_bytes(const canon_model_cfg* c, const canon_dp_plan* p) {
  std::vector<int64_t> nb;
  step_hash_sizes(c, p, nb);
  return hash_plan((int64_t)nb.size(), nb.data()).bytes;
}

// H1 of the tensors (ptrs, nbytes: host arrays) into the device digest, enqueued on s; the workspace is
// device memory of hash_plan(...).bytes bytes, 256-byte aligned.
canon_status state_hash_enqueue(int64_t n_tensors, const void* const* ptrs, const int64_t* nbytes, uint8_t* digest,
                                void* workspace, size_t workspace_bytes, hipStream_t s) {
  if (n_tensors < 0 || !digest || !workspace || (n_tensors > 0 && (!ptrs || !nbytes))) return CANON_EINVAL;
  if (n_tensors > (int64_t(1) << 24)) return CANON_EUNSUPPORTED;
  for (int64_t t = 0; t < n_tensors; ++t)
    if (nbytes[t] < 0 || (nbytes[t] > 0 && !ptrs[t])) return CANON_EINVAL;
  if ((uintptr_t)workspace & 255) return CANON_EINVAL;
  const HashPlan hp = hash_plan(n_tensors, nbytes);
  if (workspace_bytes < hp.bytes) return CANON_EWORKSPACE;
  if (hp.n_wg > INT32_MAX) return CANON_EUNSUPPORTED;
  // host tables: per tensor, and per workgroup (tensor, first leaf)
  std::vector<char> host(hp.off_la);
  HashTensor* tens = (HashTensor*)(host.data() + hp.off_tens);
  int32_t* wgt = (int32_t*)(host.data() + hp.off_wgt);
  int64_t* wgf = (int64_t*)(host.data() + hp.off_wgf);
  int64_t leaf = 0, wg = 0;
  for (int64_t t = 0; t < n_tensors; ++t) {
    const int64_t w = hash_leaf_count(nbytes[t]);
    tens[t].ptr = ptrs[t];
    tens[t].nbytes = nbytes[t];
    tens[t].leaves = w;
    tens[t].leaf_offset = leaf;
    tens[t].aligned = (((uintptr_t)ptrs[t]) & 15) == 0;
    for (int64_t f = 0; f < w; f += 256) {
      wgt[wg] = (int32_t)t;
      wgf[wg] = f;
      ++wg;
    }
    leaf += w;
  }
  char* ws = (char*)workspace;
  if (hp.off_la > 0) {
    hipError_t e = hipMemcpyAsync(ws, host.data(), hp.off_la, hipMemcpyHostToDevice, s);
    if (e != hipSuccess) return CANON_EDEVICE;
  }
  return dev(hash_launch(n_tensors, (const HashTensor*)(ws + hp.off_tens), hp.n_wg,
                         (const int32_t*)(ws + hp.off_wgt), (const int64_t*)(ws + hp.off_wgf),
                         (uint32_t*)(ws + hp.off_la), (uint32_t*)(ws + hp.off_lb), (uint32_t*)(ws + hp.off_td),
                         digest, s));
}

}  // namespace

extern "C" {

const char* canon_status_str(canon_status s) {
  switch (s) {
    case CANON_OK: return "ok";
    case CANON_EINVAL: return "invalid argument";
    case CANON_EUNSUPPORTED: return "unsupported by this version";
    case CANON_EDEVICE: return "device error";
    case CANON_EWORKSPACE: return "workspace too small";
  }
  return "unknown status";
}

int32_t canon_version(void) { return 1; }

canon_status canon_gemm_strided_batched(const canon_order* order, int32_t trans_a, int32_t trans_b, int64_t m,
                                        int64_t n, int64_t k, const uint16_t* a, int64_t lda, int64_t stride_a,
                                        const uint16_t* b, int64_t ldb, int64_t stride_b, float* c, int64_t ldc,
                                        int64_t stride_c, int64_t batch, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (m < 0 || n < 0 || k < 0 || batch < 0) return CANON_EINVAL;
  if (m == 0 || n == 0 || batch == 0) return CANON_OK;
  if (!c || (k > 0 && (!a || !b))) return CANON_EINVAL;
  if (lda < (trans_a ? m : k) || ldb < (trans_b ? k : n) || ldc < n || lda < 1 || ldb < 1) return CANON_EINVAL;
  if (batch > 65535) return CANON_EUNSUPPORTED;
  if (!gemm_k_supported(k)) return CANON_EUNSUPPORTED;
  const int64_t tiles = ((m + 63) / 64) * ((n + 127) / 128);
  if (tiles > 0x7FFFFFFF) return CANON_EUNSUPPORTED;
  GemmArgs g = mk(trans_a ? 1 : 0, trans_b ? 1 : 0, m, n, k, a, lda, b, ldb, c, ldc);
  g.batch = batch; g.nb2 = 1; g.sa1 = stride_a; g.sb1 = stride_b; g.sc1 = stride_c;
  return dev(gemm_launch(g, as_stream(stream)));
}

canon_status canon_gemm(const canon_order* order, int32_t trans_a, int32_t trans_b, int64_t m, int64_t n, int64_t k,
                        const uint16_t* a, int64_t lda, const uint16_t* b, int64_t ldb, float* c, int64_t ldc,
                        const canon_gemm_epilogue* epilogue, void* stream) {
  if (!epilogue || epilogue->kind == CANON_EPI_NONE)
    return canon_gemm_strided_batched(order, trans_a, trans_b, m, n, k, a, lda, 0, b, ldb, 0, c, ldc, 0, 1, stream);
  if (epilogue->kind != CANON_EPI_ACCUM_PLAN) return CANON_EINVAL;
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (m < 0 || n < 0 || k < 0) return CANON_EINVAL;
  if (m == 0 || n == 0) return CANON_OK;
  if (!c || (k > 0 && (!a || !b))) return CANON_EINVAL;
  if (lda < (trans_a ? m : k) || ldb < (trans_b ? k : n) || ldc < n || lda < 1 || ldb < 1) return CANON_EINVAL;
  if (!gemm_k_supported(k)) return CANON_EUNSUPPORTED;
  if (((m + 63) / 64) * ((n + 127) / 128) > 0x7FFFFFFF) return CANON_EUNSUPPORTED;
  GemmArgs g = mk(trans_a ? 1 : 0, trans_b ? 1 : 0, m, n, k, a, lda, b, ldb, c, ldc);
  g.epi = EPI_ACCUM;
  g.epi_scale = epilogue->scale;
  return dev(gemm_launch(g, as_stream(stream)));
}

canon_status canon_rownorm(const canon_order* order, int32_t dir, int64_t rows, int64_t cols, const float* x,
                           const uint16_t* gain, float eps, void* y, float* rstd, const float* dy, float* dx,
                           float* dgain, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (rows < 0 || cols < 1) return CANON_EINVAL;
  if (cols > 32768 || rows > (int64_t(1) << 26)) return CANON_EUNSUPPORTED;  // row kernels stage <= 1024 chunks
  hipStream_t s = as_stream(stream);
  if (dir == CANON_FWD || dir == CANON_FWD_F32) {
    if (rows > 0 && (!x || !gain || !y || !rstd)) return CANON_EINVAL;
    if (dir == CANON_FWD_F32) return dev(rownorm_fwd_f32_launch(rows, cols, x, gain, eps, (float*)y, rstd, s));
    return dev(rownorm_fwd_launch(rows, cols, x, gain, eps, (uint16_t*)y, rstd, s));
  }
  if (dir == CANON_BWD) {
    if (rows > 0 && (!x || !gain || !rstd || !dy || !dx)) return CANON_EINVAL;
    if (rows > 0) {  // dx is written before x, dy, rstd, gain are last read: no overlap allowed
      const char* d0 = (const char*)dx;
      const char* d1 = d0 + sizeof(float) * rows * cols;
      auto apart = [&](const void* p, size_t bytes) {
        const char* q = (const char*)p;
        return !p || q + bytes <= d0 || q >= d1;
      };
      if (!apart(x, sizeof(float) * rows * cols) || !apart(dy, sizeof(float) * rows * cols) ||
          !apart(rstd, sizeof(float) * rows) || !apart(gain, sizeof(uint16_t) * cols) ||
          !apart(dgain, sizeof(float) * cols))
        return CANON_EINVAL;
    }
    return dev(rownorm_bwd_launch(rows, cols, x, gain, rstd, dy, dx, dgain, s));
  }
  return CANON_EINVAL;
}

canon_status canon_softmax_xent(const canon_order* order, int32_t mode, int64_t rows, int64_t cols, const void* x,
                                float scale, int64_t window, const int32_t* targets, float inv_tokens, float z_loss,
                                uint16_t* out, float* row_loss, float* mean_loss, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (rows < 0 || cols < 1 || window < 0 || !(z_loss >= 0.0f) || isinf(z_loss)) return CANON_EINVAL;
  if (rows > (int64_t(1) << 31)) return CANON_EUNSUPPORTED;
  hipStream_t s = as_stream(stream);
  if (mode == CANON_SOFTMAX_CAUSAL) {
    if (cols > 32768) return CANON_EUNSUPPORTED;  // one wavefront stages at most 1024 chunks
    if (rows % cols != 0) return CANON_EINVAL;
    if (rows > 0 && (!x || !out)) return CANON_EINVAL;
    return dev(softmax_causal_launch(rows, cols, (const float*)x, scale, window, out, s));
  }
  if (mode == CANON_XENT) {
    if (rows > 0 && (!x || !targets || !out || !row_loss)) return CANON_EINVAL;
    if (rows > (int64_t(1) << 31) || cols > 131072) return CANON_EUNSUPPORTED;  // at most 4096 chunks per row
    return dev(xent_launch(rows, cols, (const uint16_t*)x, targets, inv_tokens, z_loss, out, row_loss, mean_loss,
                           s));
  }
  return CANON_EINVAL;
}

canon_status canon_grad_accum(const canon_order* order, const canon_dp_plan* plan, int64_t n,
                              const float* const* grads, float* out, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (!plan || plan->accum < 1 || plan->dp_shard < 1 || plan->dp_replicate < 1 || n < 0) return CANON_EINVAL;
  const int64_t nb = (int64_t)plan->accum * plan->dp_shard * plan->dp_replicate;
  if (nb > kMaxFusedBuffers) return CANON_EUNSUPPORTED;
  if (n == 0) return CANON_OK;
  if (!grads || !out) return CANON_EINVAL;
  PlanPtrs pp;
  memset(&pp, 0, sizeof(pp));
  for (int64_t i = 0; i < nb; ++i) {
    if (!grads[i]) return CANON_EINVAL;
    pp.p[i] = grads[i];
  }
  return dev(grad_accum_fused_launch(plan->accum, plan->dp_shard, plan->dp_replicate, n, pp, out, as_stream(stream)));
}

size_t canon_plan_state_bytes(const canon_dp_plan* plan, int64_t n) {
  if (!plan_ok(plan) || n < 0) return 0;
  return sizeof(float) * (size_t)(plan_slot_stride(n) * plan_slot_count(*plan));
}

canon_status canon_plan_begin(const canon_dp_plan* plan, int64_t n, canon_plan_cursor* cursor) {
  if (!plan_ok(plan) || n < 0 || !cursor) return CANON_EINVAL;
  if (bit_length(plan->dp_replicate) > CANON_PLAN_MAX_DEPTH) return CANON_EUNSUPPORTED;
  plan_cursor_init(*plan, n, cursor);
  return CANON_OK;
}

canon_status canon_plan_push(const canon_order* order, canon_plan_cursor* cursor, const float* grad, void* state,
                             size_t state_bytes, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (!plan_cursor_valid(cursor) || cursor->next >= plan_total(cursor->plan)) return CANON_EINVAL;
  if (cursor->n > 0 && (!grad || !state || ((uintptr_t)state & 255))) return CANON_EINVAL;
  if (state_bytes < canon_plan_state_bytes(&cursor->plan, cursor->n)) return CANON_EWORKSPACE;
  canon_plan_cursor c = *cursor;  // the caller's record changes only when every launch was enqueued
  if (plan_cursor_push(&c, (float*)state, grad, as_stream(stream)) != hipSuccess) return CANON_EDEVICE;
  *cursor = c;
  return CANON_OK;
}

canon_status canon_plan_finish(const canon_order* order, canon_plan_cursor* cursor, void* state, size_t state_bytes,
                               float* out, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (!plan_cursor_valid(cursor) || cursor->next != plan_total(cursor->plan)) return CANON_EINVAL;
  if (cursor->n > 0 && (!out || !state || ((uintptr_t)state & 255))) return CANON_EINVAL;
  if (state_bytes < canon_plan_state_bytes(&cursor->plan, cursor->n)) return CANON_EWORKSPACE;
  canon_plan_cursor c = *cursor;
  hipError_t e = hipSuccess;
  plan_cursor_finish(&c, (float*)state, out, as_stream(stream), &e);
  return dev(e);
}

canon_status canon_quant_scales(const canon_order* order, int64_t rows, int64_t cols, const uint16_t* w,
                                float* scale, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (rows < 0 || cols < 1) return CANON_EINVAL;
  if (cols > 32768 || rows > (int64_t(1) << 31)) return CANON_EUNSUPPORTED;  // one wavefront stages the row
  if (rows > 0 && (!w || !scale)) return CANON_EINVAL;
  return dev(quant_scales_launch(rows, cols, w, scale, as_stream(stream)));
}

canon_status canon_quantize(int64_t rows, int64_t cols, int32_t in_dtype, const void* x, const float* scale,
                            int32_t per_row, int8_t* q, void* stream) {
  if (rows < 0 || cols < 0 || (in_dtype != CANON_F32 && in_dtype != CANON_BF16)) return CANON_EINVAL;
  if (rows * cols > 0 && (!x || !scale || !q)) return CANON_EINVAL;
  return dev(quantize_launch(rows, cols, in_dtype, x, scale, per_row != 0, q, as_stream(stream)));
}

canon_status canon_gemm_i8(int64_t m, int64_t n, int64_t k, const int8_t* a, int64_t lda, const int8_t* b,
                           int64_t ldb, int32_t* acc, float* y, int64_t ldc, const float* sa, const float* sb,
                           void* stream) {
  if (m < 0 || n < 0 || k < 0 || lda < k || ldb < k || ldc < n) return CANON_EINVAL;
  if (k > 65536) return CANON_EUNSUPPORTED;
  if (m > 0 && n > 0 && ((k > 0 && (!a || !b)) || (!acc && !y) || (y && (!sa || !sb)))) return CANON_EINVAL;
  GemmI8Args g{};
  g.a = a; g.b = b; g.acc = acc; g.y = y; g.sa = sa; g.sb = sb;
  g.m = m; g.n = n; g.k = k; g.lda = lda; g.ldb = ldb; g.ldc = ldc;
  return dev(gemm_i8_launch(g, as_stream(stream)));
}

canon_status canon_qlinear_bwd(const canon_order* order, int64_t T, int64_t N, int64_t K, const float* dy,
                               const int8_t* qx, const float* sx, const int8_t* qw, const float* sw, float* dx,
                               float* dw, void* workspace, size_t workspace_bytes, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (T < 1 || N < 1 || K < 1 || (!dx && !dw)) return CANON_EINVAL;
  if ((dx && N % 256) || (dw && T % 256)) return CANON_EUNSUPPORTED;  // whole rotation blocks
  if ((dx && N > 65536) || (dw && T > 65536)) return CANON_EUNSUPPORTED;  // the int8 GEMM's k bound
  if (T * N > (int64_t(1) << 34) || K * (N > T ? N : T) > (int64_t(1) << 34)) return CANON_EUNSUPPORTED;
  if (!dy || !qx || !sx || !qw || !sw || !workspace) return CANON_EINVAL;
  if (workspace_bytes < qlinear_bwd_workspace_bytes(T, N, K)) return CANON_EWORKSPACE;
  if (((uintptr_t)dy & 15) || ((uintptr_t)workspace & 255)) return CANON_EINVAL;
  return dev(qlinear_bwd_launch(T, N, K, dy, 0, qx, sx, qw, sw, dx, dw, workspace, as_stream(stream)));
}

size_t canon_qlinear_bwd_workspace_bytes(int64_t T, int64_t N, int64_t K) {
  if (T < 1 || N < 1 || K < 1) return 0;
  return qlinear_bwd_workspace_bytes(T, N, K);
}


size_t canon_state_hash_workspace_bytes(int64_t n_tensors, const int64_t* nbytes) {
  if (n_tensors < 0 || (n_tensors > 0 && !nbytes)) return 0;
  for (int64_t t = 0; t < n_tensors; ++t)
    if (nbytes[t] < 0) return 0;
  return hash_plan(n_tensors, nbytes).bytes;
}

canon_status canon_state_hash(int64_t n_tensors, const void* const* ptrs, const int64_t* nbytes, uint8_t* digest,
                              void* workspace, size_t workspace_bytes, void* stream) {
  return state_hash_enqueue(n_tensors, ptrs, nbytes, digest, workspace, workspace_bytes, as_stream(stream));
}

canon_status canon_adamw(int64_t n_tensors, const int64_t* sizes, uint16_t* const* params, float* const* m,
                         float* const* v, const float* const* grads, const uint8_t* decay_mask,
                         const canon_adamw_consts* consts, void* stream) {
  if (n_tensors < 0 || !consts) return CANON_EINVAL;
  if (n_tensors > 0 && (!sizes || !params || !m || !v || !grads || !decay_mask)) return CANON_EINVAL;
  for (int64_t t = 0; t < n_tensors; ++t) {
    if (sizes[t] < 0) return CANON_EINVAL;
    if (sizes[t] > 0 && (!params[t] || !m[t] || !v[t] || !grads[t])) return CANON_EINVAL;
  }
  const float c9[9] = {consts->lr, consts->beta1, consts->one_minus_beta1, consts->beta2, consts->one_minus_beta2,
                       consts->inv_bc1, consts->inv_bc2, consts->eps, consts->decay_factor};
  for (int64_t t = 0; t < n_tensors; ++t) {
    hipError_t e = adamw_launch(sizes[t], params[t], m[t], v[t], grads[t], decay_mask[t] != 0, c9, nullptr,
                                nullptr, as_stream(stream));
    if (e != hipSuccess) return CANON_EDEVICE;
  }
  return CANON_OK;
}

size_t canon_clip_grad_norm_workspace_bytes(int64_t n_tensors, const int64_t* sizes) {
  if (n_tensors < 0 || (n_tensors > 0 && !sizes)) return 0;
  int64_t n = 0;
  for (int64_t t = 0; t < n_tensors; ++t) {
    if (sizes[t] < 0) return 0;
    n += sizes[t];
  }
  Carver cv(nullptr);
  cv.take<const float*>(n_tensors);
  cv.take<int64_t>(n_tensors + 1);
  cv.take<float>(gnorm_blocks(n));
  cv.take<float>(1);
  return cv.off + 256;
}

canon_status canon_clip_grad_norm(const canon_order* order, int64_t n_tensors, const int64_t* sizes,
                                  float* const* grads, const canon_clip* clip, void* workspace,
                                  size_t workspace_bytes, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (n_tensors < 0 || !clip || (n_tensors > 0 && (!sizes || !grads))) return CANON_EINVAL;
  if (!(clip->max_norm > 0.0f) || clip->skip_steps < 0 || (clip->skip_steps > 0 && !clip->skip_state))
    return CANON_EINVAL;
  if (n_tensors > INT32_MAX - 1) return CANON_EUNSUPPORTED;
  int64_t n = 0;
  bool vec4 = true;
  for (int64_t t = 0; t < n_tensors; ++t) {
    if (sizes[t] < 0 || (sizes[t] > 0 && !grads[t])) return CANON_EINVAL;
    n += sizes[t];
    if (sizes[t] % 4 != 0 || ((uintptr_t)grads[t] & 15)) vec4 = false;
  }
  if (n > (int64_t(1) << 40)) return CANON_EUNSUPPORTED;
  const size_t need = canon_clip_grad_norm_workspace_bytes(n_tensors, sizes);
  if (!workspace || workspace_bytes < need) return CANON_EWORKSPACE;
  hipStream_t s = as_stream(stream);
  Carver cv(workspace);
  const float** ptr_d = cv.take<const float*>(n_tensors);
  int64_t* start_d = cv.take<int64_t>(n_tensors + 1);
  float* part = cv.take<float>(gnorm_blocks(n));
  float* coef = cv.take<float>(1);
  NormSrc src{};
  src.nt = (int32_t)n_tensors;
  if (n_tensors == 1) {
    src.one = grads[0];
  } else if (n_tensors > 1) {
    std::vector<const float*> hp(grads, grads + n_tensors);
    std::vector<int64_t> hs(n_tensors + 1, 0);
    for (int64_t t = 0; t < n_tensors; ++t) hs[t + 1] = hs[t] + sizes[t];
    TRY(hipMemcpyAsync(ptr_d, hp.data(), sizeof(float*) * n_tensors, hipMemcpyHostToDevice, s));
    TRY(hipMemcpyAsync(start_d, hs.data(), sizeof(int64_t) * (n_tensors + 1), hipMemcpyHostToDevice, s));
    src.ptr = ptr_d;
    src.start = start_d;
  }
  ClipDecision d{};
  d.max_norm = clip->max_norm;
  d.spike_norm = clip->spike_norm;
  d.skip_steps = clip->skip_steps;
  d.norm_out = clip->norm_out;
  d.coef_out = coef;
  d.skip_state = clip->skip_state;
  d.skipped_out = clip->skipped_out;
  TRY(gnorm_launch(src, n, vec4 ? 1 : 0, part, d, s));
  for (int64_t t = 0; t < n_tensors; ++t) TRY(clip_scale_launch(sizes[t], grads[t], coef, s));
  return CANON_OK;
}

size_t canon_attn_pv_i8_workspace_bytes(int64_t batch, int64_t n_kv_heads, int64_t seq, int64_t head_dim) {
  if (batch < 1 || n_kv_heads < 1 || seq < 1 || head_dim < 1) return 0;
  const int64_t nb = attn_pv_blocks(seq);
  Carver cv(nullptr);
  cv.take<int8_t>(batch * n_kv_heads * head_dim * nb * 64);
  cv.take<float>(batch * n_kv_heads * nb);
  return cv.off + 256;
}

canon_status canon_attn_pv_i8(int64_t batch, int64_t n_heads, int64_t n_kv_heads, int64_t seq, int64_t head_dim,
                              int64_t window, const uint16_t* P, const uint16_t* V, float* o_f32, uint16_t* o_bf16,
                              void* workspace, size_t workspace_bytes, void* stream) {
  if (batch < 0 || n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads != 0 || seq < 1 || head_dim < 1 ||
      window < 0)
    return CANON_EINVAL;
  if (head_dim % 32 != 0 || head_dim > 256 || seq > 8192 || batch * n_heads > 65535) return CANON_EUNSUPPORTED;
  if (batch == 0) return CANON_OK;
  if (!P || !V || (!o_f32 && !o_bf16) || !workspace || ((uintptr_t)workspace & 255)) return CANON_EINVAL;
  if (workspace_bytes < canon_attn_pv_i8_workspace_bytes(batch, n_kv_heads, seq, head_dim)) return CANON_EWORKSPACE;
  const int64_t nb = attn_pv_blocks(seq);
  Carver cv(workspace);
  int8_t* qvt = cv.take<int8_t>(batch * n_kv_heads * head_dim * nb * 64);
  float* sv = cv.take<float>(batch * n_kv_heads * nb);
  return dev(attn_pv_i8_launch(batch, n_heads, n_kv_heads, seq, head_dim, window, P, V, o_f32, o_bf16,
                               n_heads * head_dim, qvt, sv, as_stream(stream)));
}

canon_status canon_attn_dq_fixed(int64_t batch, int64_t n_heads, int64_t n_kv_heads, int64_t seq, int64_t head_dim,
                                 int64_t window, int32_t frac_bits, const uint16_t* dS, const uint16_t* K, float* dQ,
                                 void* stream) {
  if (batch < 0 || n_heads < 1 || n_kv_heads < 1 || n_heads % n_kv_heads != 0 || seq < 1 || head_dim < 1 ||
      window < 0 || frac_bits < 1 || frac_bits > 62)
    return CANON_EINVAL;
  if ((head_dim != 16 && head_dim != 32 && head_dim != 64 && head_dim != 128) || batch * n_heads > 65535)
    return CANON_EUNSUPPORTED;
  if (batch == 0) return CANON_OK;
  if (!dS || !K || !dQ) return CANON_EINVAL;
  return dev(attn_dq_fixed_launch(batch, n_heads, n_kv_heads, seq, head_dim, window, frac_bits, dS, K, dQ,
                                  n_heads * head_dim, as_stream(stream)));
}

size_t canon_lsq_step_grad_workspace_bytes(int64_t T, int64_t K) {
  if (T < 0 || K < 1) return 0;
  return sizeof(float) * (size_t)(lsq_grad_parts(T * K) + 1) + 256;
}

canon_status canon_lsq_step_grad(const canon_order* order, int64_t T, int64_t K, const uint16_t* x, const float* s,
                                 const float* dx, float* grad, void* workspace, size_t workspace_bytes, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (T < 0 || K < 1 || !s || !grad || (T > 0 && (!x || !dx))) return CANON_EINVAL;
  if (T * K > (int64_t(1) << 40)) return CANON_EUNSUPPORTED;
  if (!workspace || workspace_bytes < canon_lsq_step_grad_workspace_bytes(T, K)) return CANON_EWORKSPACE;
  return dev(lsq_grad_launch(T * K, x, s, dx, lsq_gamma(K), (float*)workspace, grad, as_stream(stream)));
}

size_t canon_embed_bwd_workspace_bytes(int64_t T, int64_t d) {
  if (T < 0 || d < 1 || T >= (int64_t(1) << 25)) return 0;
  return embed_bwd_scratch_bytes(T, d) + 256;
}

canon_status canon_embed_bwd(const canon_order* order, int64_t T, int64_t V, int64_t d, const int32_t* tokens,
                             const float* dx, float* dE, void* workspace, size_t workspace_bytes, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (T < 0 || V < 1 || d < 1 || !dE || (T > 0 && (!tokens || !dx))) return CANON_EINVAL;
  if (T >= (int64_t(1) << 25) || V > (int64_t(1) << 31) - 1) return CANON_EUNSUPPORTED;
  const size_t need = canon_embed_bwd_workspace_bytes(T, d);
  if (!workspace || workspace_bytes < need) return CANON_EWORKSPACE;
  void* ws = (void*)(((uintptr_t)workspace + 255) & ~(uintptr_t)255);
  return dev(embed_bwd_launch(1, T, d, tokens, T, V, dx, dE, ws, as_stream(stream)));
}

canon_status canon_lsq_step_grad_noalloc(const canon_order* order, int64_t T, int64_t K, const uint16_t* x,
                                         const float* s, const float* dx, float* grad, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (T < 0 || K < 1 || !s || !grad || (T > 0 && (!x || !dx))) return CANON_EINVAL;
  if (T > lsq_noalloc_max_terms() / K) return CANON_EUNSUPPORTED;  // T K beyond the library's array
  float* part = nullptr;
  TRY(lsq_scratch(&part));
  return dev(lsq_grad_launch(T * K, x, s, dx, lsq_gamma(K), part, grad, as_stream(stream)));
}

int64_t canon_lsq_step_grad_noalloc_max_terms(void) { return lsq_noalloc_max_terms(); }

canon_status canon_devmath(int32_t op, int64_t n, const float* a, const float* b, const float* c, float* out,
                           void* stream) {
  if (op < 0 || op > 10 || n < 0) return CANON_EINVAL;
  if (n == 0) return CANON_OK;
  if (!a || !out) return CANON_EINVAL;
  if ((op <= 4 && !b) || (op == 3 && !c)) return CANON_EINVAL;
  return dev(devmath_launch(op, n, a, b, c, out, as_stream(stream)));
}

size_t canon_block_workspace_bytes(const canon_model_cfg* cfg, int32_t batch) {
  if (!cfg_ok(cfg) || batch < 1) return 0;
  Dims D = dims_of(cfg, batch);
  Carver cv(nullptr);
  LayerSave sv;
  Scratch sc;
  carve_save(cv, D, sv);
  carve_scratch(cv, D, sc);
  return cv.off + 256;
}

canon_status canon_block_fwd_bwd(const canon_order* order, const canon_model_cfg* cfg, int32_t batch, const float* x,
                                 const float* dy, const uint16_t* const* w, const float* rope_cos,
                                 const float* rope_sin, float* y, float* dx, float* const* dw, void* workspace,
                                 size_t workspace_bytes, void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (!cfg_ok(cfg) || batch < 1 || !x || !dy || !w || !rope_cos || !rope_sin || !y || !dx || !dw)
    return CANON_EINVAL;
  if (!variants_supported(cfg, (int64_t)batch * cfg->seq)) return CANON_EUNSUPPORTED;
  const int nw = cfg->int8_linear ? 10 : 6;
  for (int i = 0; i < nw; ++i)
    if (!w[i] || !dw[i]) return CANON_EINVAL;
  if ((int64_t)batch * cfg->n_heads > 65535) return CANON_EUNSUPPORTED;
  const size_t need = canon_block_workspace_bytes(cfg, batch);
  if (!workspace || workspace_bytes < need) return CANON_EWORKSPACE;
  Dims D = dims_of(cfg, batch);
  Carver cv(workspace);
  LayerSave sv;
  Scratch sc;
  carve_save(cv, D, sv);
  carve_scratch(cv, D, sc);
  hipStream_t s = as_stream(stream);
  if (D.int8 && (st = prep_int8_layer(D, w, sv, s)) != CANON_OK) return st;
  st = block_forward(D, w, rope_cos, rope_sin, x, sv, sc, y, s);
  if (st != CANON_OK) return st;
  return block_backward(D, w, rope_cos, rope_sin, x, sv, sc, dy, dx, dw, s);
}

size_t canon_step_workspace_bytes(const canon_model_cfg* cfg, const canon_dp_plan* plan) {
  if (!cfg_ok(cfg) || !plan || plan->accum < 1 || plan->dp_shard < 1 || plan->dp_replicate < 1) return 0;
  std::vector<int64_t> sz;
  std::vector<uint8_t> decay;
  tensor_sizes(cfg, sz, decay);
  int64_t P = 0;
  for (int64_t v : sz) P += v;
  Carver cv(nullptr);
  StepLayout L;
  carve_step(cv, cfg, plan, P, L);
  return cv.off + 256;
}

canon_status canon_step(const canon_order* order, const canon_model_cfg* cfg, const canon_dp_plan* plan,
                        uint16_t* const* params, float* const* m, float* const* v, int32_t step_t,
                        const int32_t* windows, const float* rope_cos, const float* rope_sin,
                        const canon_adamw_consts* consts, const canon_clip* clip, void* workspace,
                        size_t workspace_bytes, float* loss_out, float* const* grads_out, uint8_t* state_digest,
                        void* stream) {
  canon_status st = check_order(order);
  if (st != CANON_OK) return st;
  if (step_t < 1) return CANON_EINVAL;  // AdamW's step index starts at 1
  if (!cfg_ok(cfg) || !plan || plan->accum < 1 || plan->dp_shard < 1 || plan->dp_replicate < 1) return CANON_EINVAL;
  if (!params || !m || !v || !windows || !rope_cos || !rope_sin || !consts || !loss_out) return CANON_EINVAL;
  if (!variants_supported(cfg, (int64_t)cfg->micro_seqs * cfg->seq)) return CANON_EUNSUPPORTED;
  if (clip && (!(clip->max_norm > 0.0f) || clip->skip_steps < 0 || (clip->skip_steps > 0 && !clip->skip_state)))
    return CANON_EINVAL;
  std::vector<int64_t> sz;
  std::vector<uint8_t> decay;
  tensor_sizes(cfg, sz, decay);
  const int64_t nt = (int64_t)sz.size();
  for (int64_t t = 0; t < nt; ++t)
    if (!params[t] || !m[t] || !v[t] || (grads_out && !grads_out[t])) return CANON_EINVAL;
  if ((int64_t)cfg->micro_seqs * cfg->n_heads > 65535) return CANON_EUNSUPPORTED;
  std::vector<int64_t> off(nt + 1, 0);
  for (int64_t t = 0; t < nt; ++t) off[t + 1] = off[t] + sz[t];
  const int64_t P = off[nt];
  const size_t need = canon_step_workspace_bytes(cfg, plan);
  if (!workspace || workspace_bytes < need) return CANON_EWORKSPACE;
  if (state_digest && ((uintptr_t)workspace & 255)) return CANON_EINVAL;  // the hash's tables are aligned

  hipStream_t s = as_stream(stream);
  Carver cv(workspace);
  StepLayout L;
  carve_step(cv, cfg, plan, P, L);
  const Dims D = dims_of(cfg, cfg->micro_seqs);
  const int R = plan->dp_shard * plan->dp_replicate;
  const int64_t S1 = cfg->seq + 1, mb = cfg->micro_seqs;
  const int64_t M = (int64_t)R * plan->accum * mb;
  const float invT = (float)(1.0 / (double)D.T);

  TRY(hipMemsetAsync(L.bad, 0, sizeof(int32_t), s));
  TRY(token_check_launch(M * S1, windows, cfg->vocab, L.bad, s));

  canon_plan_cursor gplan, lplan;
  plan_cursor_init(*plan, P, &gplan);
  plan_cursor_init(*plan, 1, &lplan);
  const int nl = cfg->n_layers;
  const int64_t l0 = cfg->embed_norm ? 2 : 1;  // first layer tensor
  const int PL = cfg->int8_linear ? 10 : 6;    // tensors per layer
  if (cfg->int8_linear)  // the weights' codes and re-pinned steps, once per step
    for (int l = 0; l < nl; ++l) {
      const uint16_t* w[10];
      for (int i = 0; i < PL; ++i) w[i] = params[l0 + PL * l + i];
      if ((st = prep_int8_layer(D, w, L.saves[l], s)) != CANON_OK) return st;
    }
  for (int r = 0; r < R; ++r) {
    for (int k = 0; k < plan->accum; ++k) {
      // R12: windows r + R*(k*mb + s), s < mb
      for (int64_t si = 0; si < mb; ++si) {
        const int64_t mw = r + (int64_t)R * (k * mb + si);
        TRY(hipMemcpyAsync(L.win + si * S1, windows + mw * S1, sizeof(int32_t) * S1, hipMemcpyDeviceToDevice, s));
      }
      if (cfg->embed_norm) {  // the embedding norm's fp32 output is the first block's input
        TRY(embed_gather_launch(mb, D.S, D.d, L.win, S1, params[0], D.V, L.x_emb, s));
        TRY(rownorm_fwd_f32_launch(D.T, D.d, L.x_emb, params[1], D.eps, L.xs[0], L.rstd_emb, s));
      } else {
        TRY(embed_gather_launch(mb, D.S, D.d, L.win, S1, params[0], D.V, L.xs[0], s));
      }
      TRY(labels_launch(mb, D.S, L.win, S1, L.lab, s));
      for (int l = 0; l < nl; ++l) {
        const uint16_t* w[10];
        for (int i = 0; i < PL; ++i) w[i] = params[l0 + PL * l + i];
        Dims Dl = D;
        Dl.window = layer_window(cfg, l);
        st = block_forward(Dl, w, rope_cos, rope_sin, L.xs[l], L.saves[l], L.sc, L.xs[l + 1], s);
        if (st != CANON_OK) return st;
      }
      const int64_t i_fn = l0 + PL * nl, i_head = i_fn + 1;
      TRY(rownorm_fwd_launch(D.T, D.d, L.xs[nl], params[i_fn], D.eps, L.xf, L.rstdf, s));
      TRY(gemm(mk(0, 1, D.T, D.V, D.d, L.xf, D.d, params[i_head], D.d, L.logits, D.V, 1), s));
      TRY(xent_launch(D.T, D.V, L.logits, L.lab, invT, D.z_loss, L.dlogits, L.row_loss, L.loss_mb, s));
      TRY(gemm(mk(1, 0, D.V, D.d, D.T, L.dlogits, D.V, L.xf, D.d, L.grad + off[i_head], D.d), s));
      TRY(gemm(mk(0, 0, D.T, D.d, D.V, L.dlogits, D.V, params[i_head], D.d, L.dxf, D.d), s));
      TRY(rownorm_bwd_launch(D.T, D.d, L.xs[nl], params[i_fn], L.rstdf, L.dxf, L.dxA, L.grad + off[i_fn], s));
      float* dcur = L.dxA;
      float* dnext = L.dxB;
      for (int l = nl - 1; l >= 0; --l) {
        const uint16_t* w[10];
        float* dw[10];
        for (int i = 0; i < PL; ++i) {
          w[i] = params[l0 + PL * l + i];
          dw[i] = L.grad + off[l0 + PL * l + i];
        }
        Dims Dl = D;
        Dl.window = layer_window(cfg, l);
        st = block_backward(Dl, w, rope_cos, rope_sin, L.xs[l], L.saves[l], L.sc, dcur, dnext, dw, s);
        if (st != CANON_OK) return st;
        float* t = dcur; dcur = dnext; dnext = t;
      }
      if (cfg->embed_norm) {  // back through the embedding norm to the gathered rows
        TRY(rownorm_bwd_launch(D.T, D.d, L.x_emb, params[1], L.rstd_emb, dcur, dnext, L.grad + off[1], s));
        float* t = dcur; dcur = dnext; dnext = t;
      }
      TRY(embed_bwd_launch(mb, D.S, D.d, L.win, S1, D.V, dcur, L.grad + off[0], L.embed_scratch, s));
      TRY(plan_cursor_push(&gplan, L.plan_slots, L.grad, s));
      TRY(plan_cursor_push(&lplan, L.loss_slots, L.loss_mb, s));
    }
  }
  hipError_t e = hipSuccess;
  float* g = plan_cursor_finish(&gplan, L.plan_slots, nullptr, s, &e);
  TRY(e);
  plan_cursor_finish(&lplan, L.loss_slots, loss_out, s, &e);
  TRY(e);
  TRY(set_nan_if_launch(L.bad, loss_out, s));
  if (grads_out)
    for (int64_t t = 0; t < nt; ++t)
      TRY(hipMemcpyAsync(grads_out[t], g + off[t], sizeof(float) * sz[t], hipMemcpyDeviceToDevice, s));
  const float c9[9] = {consts->lr, consts->beta1, consts->one_minus_beta1, consts->beta2, consts->one_minus_beta2,
                       consts->inv_bc1, consts->inv_bc2, consts->eps, consts->decay_factor};
  const float* gscale = nullptr;
  const int32_t* skip = L.bad;
  if (clip) {
    // R15 on the reduced gradient (one flat buffer in declared order): pre-clip norm, clip coefficient and
    // spike counter; the clip itself is applied inside AdamW
    NormSrc src{};
    src.one = g;
    src.nt = 1;
    ClipDecision d{};
    d.max_norm = clip->max_norm;
    d.spike_norm = clip->spike_norm;
    d.skip_steps = clip->skip_steps;
    d.bad = L.bad;
    d.norm_out = clip->norm_out;
    d.coef_out = L.clip_coef;
    d.skip_state = clip->skip_state;
    d.skip_flag = L.skip;
    d.skipped_out = clip->skipped_out;
    TRY(gnorm_launch(src, P, (P % 4 == 0 && ((uintptr_t)g & 15) == 0) ? 1 : 0, L.norm_part, d, s));
    gscale = L.clip_coef;
    skip = L.skip;
  }
  for (int64_t t = 0; t < nt; ++t)
    TRY(adamw_launch(sz[t], params[t], m[t], v[t], g + off[t], decay[t], c9, gscale, skip, s));
  if (state_digest) {  // the per-step audit hash of the state this step leaves
    std::vector<int64_t> nb;
    step_hash_sizes(cfg, plan, nb);
    std::vector<const void*> ptrs;
    ptrs.push_back(windows);
    for (int64_t t = 0; t < nt; ++t) ptrs.push_back(params[t]);
    for (int64_t t = 0; t < nt; ++t) ptrs.push_back(m[t]);
    for (int64_t t = 0; t < nt; ++t) ptrs.push_back(v[t]);
    for (int64_t t = 0; t < nt; ++t) ptrs.push_back(g + off[t]);
    st = state_hash_enqueue((int64_t)nb.size(), ptrs.data(), nb.data(), state_digest, L.hash_ws,
                            step_hash_bytes(cfg, plan), s);
    if (st != CANON_OK) return st;
  }
  return CANON_OK;
}

}  // extern "C"
