// gemm.hip - canonical-order GEMM (R1, R2) on gfx950 matrix cores.
//
// C[i,j] = sum_k A(i,k) B(k,j): the k terms form chunks of 32; each chunk is a left-to-right chain of
// fused multiply-adds from +0 in ascending k; the chunk partials are combined by the binary-carry fold of
// Algorithm 2 (pushed in ascending chunk order, leftover blocks combined smallest first).
//
// Matrix-core mapping.  v_mfma_f32_32x32x1_2b_f32 performs, for two independent 32x32 blocks, the
// rank-1 update D = C + a*b with ONE product per output element.  On gfx950 it returns RN(c + a*b) with
// the flush rule of R0, bit for bit (checked against a sequential fma chain, including ties, signed zeros
// and 32-step dependent chains).  A bf16 x bf16 product is exact in fp32, so a chain of these updates,
// one per k, is exactly the canonical fma chain.  The bf16 MFMA shapes that sum several products inside
// one instruction do not give the chain's roundings and are not used.
//
// Tiling: a workgroup of 4 waves computes a 64 x 128 tile of C; wave (wr, wc) owns rows 32*wr..+32 and
// columns 64*wc..+64 as the instruction's two 32x32 blocks (block 0: columns +0..31, block 1: +32..63).
// Per chunk the 64x32 A tile and 32x128 B tile are staged through LDS as fp32 (widened once, k-major so
// that a lane reads one float per k), double buffered, with the next chunk's global loads issued before
// the current chunk's MFMA chain.  The binary-carry stack lives in registers (MAXL levels of 32 floats).
//
// Causal modes (attention): KMODE_TRAIL skips key chunks that are masked for every row of the tile and
// KMODE_LEAD skips query chunks below the tile; the skipped chunks' partials are exactly +0 in the
// canonical chain and are still folded (pushed as +0), so the result equals the full-range chain.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

typedef float v32f __attribute__((ext_vector_type(32)));

constexpr int BM = 64, BN = 128, KC = 32;
constexpr int APAD = 4, BPAD = 4;

template <bool TA, bool TB>
__device__ __forceinline__ void load_tiles(const GemmArgs& g, const uint16_t* A, const uint16_t* B, int64_t row0,
                                           int64_t col0, int64_t k0, uint16_t (&ra)[8], uint16_t (&rb)[16]) {
  const int t = threadIdx.x;
  // A: 64 rows x 32 k, 8 consecutive elements per thread
  {
    int64_t r, kk;
    if (!TA) { r = t >> 2; kk = (t & 3) * 8; }
    else { kk = t >> 3; r = (t & 7) * 8; }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      int64_t ri = row0 + r + (TA ? e : 0), ki = k0 + kk + (TA ? 0 : e);
      ra[e] = (ri < g.m && ki < g.k) ? (TA ? A[ki * g.lda + ri] : A[ri * g.lda + ki]) : (uint16_t)0;
    }
  }
  // B: 32 k x 128 cols, two groups of 8 per thread
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    int idx = t + 256 * it;
    int64_t c, kk;
    if (!TB) { kk = idx >> 4; c = (idx & 15) * 8; }
    else { c = idx >> 2; kk = (idx & 3) * 8; }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      int64_t ci = col0 + c + (TB ? 0 : e), ki = k0 + kk + (TB ? e : 0);
      rb[it * 8 + e] = (ci < g.n && ki < g.k) ? (TB ? B[ci * g.ldb + ki] : B[ki * g.ldb + ci]) : (uint16_t)0;
    }
  }
}

template <bool TA, bool TB>
__device__ __forceinline__ void store_tiles(float (*As)[BM + APAD], float (*Bs)[BN + BPAD], const uint16_t (&ra)[8],
                                            const uint16_t (&rb)[16]) {
  const int t = threadIdx.x;
  {
    int r, kk;
    if (!TA) { r = t >> 2; kk = (t & 3) * 8; }
    else { kk = t >> 3; r = (t & 7) * 8; }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (!TA) As[kk + e][r] = bf16_to_f32(ra[e]);
      else As[kk][r + e] = bf16_to_f32(ra[e]);
    }
  }
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    int idx = t + 256 * it;
    int c, kk;
    if (!TB) { kk = idx >> 4; c = (idx & 15) * 8; }
    else { c = idx >> 2; kk = (idx & 3) * 8; }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if (!TB) Bs[kk][c + e] = bf16_to_f32(rb[it * 8 + e]);
      else Bs[kk + e][c] = bf16_to_f32(rb[it * 8 + e]);
    }
  }
}

// Binary-carry stack of Algorithm 2 with MAXL levels, each level a register set of its own (a recursive
// member chain, so no level is ever addressed dynamically).  push(p, c) pushes the partial of chunk c
// (c = number of partials pushed before it): at each level whose bit of c is set the stored block is
// merged, earlier block on the left, and the carry moves up.  The caller keeps the chunk count below
// 2^MAXL so a carry never leaves the top level.
template <int L>
struct FoldStack {
  v32f s;
  FoldStack<L - 1> up;
  __device__ __forceinline__ void clear(const v32f& z) { s = z; up.clear(z); }
  __device__ __forceinline__ void push(v32f p, int64_t c) {
    if (c & 1) up.push(s + p, c >> 1);
    else s = p;
  }
  // Result: lowest occupied level first, then the others in ascending level order
  __device__ __forceinline__ void result(v32f& r, bool& have, int64_t n) const {
    if (n & 1) {
      if (!have) { r = s; have = true; }
      else r = s + r;
    }
    up.result(r, have, n >> 1);
  }
};
template <>
struct FoldStack<0> {
  __device__ __forceinline__ void clear(const v32f&) {}
  __device__ __forceinline__ void push(v32f, int64_t) {}
  __device__ __forceinline__ void result(v32f&, bool&, int64_t) const {}
};

template <int MAXL, bool TA, bool TB>
__global__ __launch_bounds__(256) void gemm_mfma_kernel(GemmArgs g) {
  __shared__ float As[2][KC][BM + APAD];
  __shared__ float Bs[2][KC][BN + BPAD];

  const int64_t tiles_n = (g.n + BN - 1) / BN;
  const int64_t tm = blockIdx.x / tiles_n, tn = blockIdx.x % tiles_n;
  const int64_t row0 = tm * BM, col0 = tn * BN;
  if (g.tri_lower && col0 > row0 + BM - 1) return;  // output tile entirely above the diagonal

  const int64_t z = blockIdx.z;
  const int64_t z1 = z / g.nb2, z2 = z % g.nb2;
  const uint16_t* A = g.a + z1 * g.sa1 + z2 * g.sa2;
  const uint16_t* B = g.b + z1 * g.sb1 + z2 * g.sb2;

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;

  const int64_t nc = (g.k + KC - 1) / KC;
  int64_t c_begin = 0, c_end = nc;
  if (g.kmode == KMODE_TRAIL) {
    int64_t last_row = row0 + BM < g.m ? row0 + BM : g.m;  // rows of this tile are < last_row
    int64_t ce = (last_row + KC - 1) / KC;
    c_end = ce < nc ? ce : nc;
  } else if (g.kmode == KMODE_LEAD) {
    int64_t cb = row0 / KC;
    c_begin = cb < nc ? cb : nc;
  }

  v32f zero;
#pragma unroll
  for (int v = 0; v < 32; ++v) zero[v] = 0.0f;
  // leading skipped chunks: the stack after pushing c_begin partials of +0 holds +0 at its set bits
  FoldStack<MAXL> S;
  S.clear(zero);

  uint16_t ra[8], rb[16];
  int buf = 0;
  if (c_begin < c_end) {
    load_tiles<TA, TB>(g, A, B, row0, col0, c_begin * KC, ra, rb);
    store_tiles<TA, TB>(As[0], Bs[0], ra, rb);
  }
  __syncthreads();

  const int arow = wr * 32 + (lane & 31);
  const int bcol = wc * 64 + lane;
  for (int64_t c = c_begin; c < c_end; ++c) {
    const bool more = c + 1 < c_end;
    if (more) load_tiles<TA, TB>(g, A, B, row0, col0, (c + 1) * KC, ra, rb);
    v32f acc = zero;
    const int64_t kleft = g.k - c * KC;
    if (kleft >= KC) {
#pragma unroll
      for (int kk = 0; kk < KC; ++kk)
        acc = __builtin_amdgcn_mfma_f32_32x32x1f32(As[buf][kk][arow], Bs[buf][kk][bcol], acc, 0, 0, 0);
    } else {
      for (int kk = 0; kk < (int)kleft; ++kk)
        acc = __builtin_amdgcn_mfma_f32_32x32x1f32(As[buf][kk][arow], Bs[buf][kk][bcol], acc, 0, 0, 0);
    }
    S.push(acc, c);
    if (more) store_tiles<TA, TB>(As[buf ^ 1], Bs[buf ^ 1], ra, rb);
    __syncthreads();
    buf ^= 1;
  }
  // trailing skipped chunks: push +0 partials (their merges turn a -0 partial into +0, as the chain does)
  for (int64_t c = c_end; c < nc; ++c) S.push(zero, c);

  v32f r = zero;
  bool have = false;
  S.result(r, have, nc);

  // store: register v, lane l -> block v/16, row (v%4) + 4*(l/32) + 8*((v%16)/4), column l%32
  const int64_t crow0 = row0 + wr * 32, ccol0 = col0 + wc * 64;
#pragma unroll
  for (int v = 0; v < 32; ++v) {
    const int vv = v & 15, blk = v >> 4;
    const int64_t i = crow0 + (vv & 3) + 4 * (lane >> 5) + 8 * (vv >> 2);
    const int64_t j = ccol0 + blk * 32 + (lane & 31);
    if (i < g.m && j < g.n) {
      if (g.out_bf16) {
        uint16_t* C = (uint16_t*)g.c + z1 * g.sc1 + z2 * g.sc2;
        C[i * g.ldc + j] = f32_to_bf16(r[v]);
      } else {
        float* C = (float*)g.c + z1 * g.sc1 + z2 * g.sc2;
        C[i * g.ldc + j] = r[v];
      }
    }
  }
}

template <int MAXL>
static hipError_t launch_maxl(const GemmArgs& g, dim3 grid, hipStream_t s) {
  if (!g.trans_a && !g.trans_b) hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, false, false>), grid, dim3(256), 0, s, g);
  else if (!g.trans_a && g.trans_b) hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, false, true>), grid, dim3(256), 0, s, g);
  else if (g.trans_a && !g.trans_b) hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, true, false>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, true, true>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

int gemm_max_levels() { return 12; }

hipError_t gemm_launch(const GemmArgs& g, hipStream_t s) {
  if (g.m == 0 || g.n == 0 || g.batch == 0) return hipSuccess;
  const int64_t nc = (g.k + KC - 1) / KC;
  int bits = 0;
  while ((int64_t(1) << bits) <= nc) ++bits;  // nc < 2^bits: a push never runs past the top level
  const int64_t tiles = ((g.m + BM - 1) / BM) * ((g.n + BN - 1) / BN);
  dim3 grid((unsigned)tiles, 1, (unsigned)g.batch);
  if (bits <= 3) return launch_maxl<3>(g, grid, s);
  if (bits <= 5) return launch_maxl<5>(g, grid, s);
  if (bits <= 7) return launch_maxl<7>(g, grid, s);
  if (bits <= 9) return launch_maxl<9>(g, grid, s);
  if (bits <= 11) return launch_maxl<11>(g, grid, s);
  if (bits <= 12) return launch_maxl<12>(g, grid, s);
  return hipErrorInvalidValue;
}

}  // namespace canon
