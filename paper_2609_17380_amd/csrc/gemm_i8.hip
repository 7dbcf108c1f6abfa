// gemm_i8.hip - exact int8 GEMM on the int8 matrix cores, with the dequantisation epilogue of the int8
// quantised linear.
//
// acc[i][j] = sum over k of a[i][k] * b[j][k] with int8 operands (a [m][k], b [n][k], both k-contiguous,
// b holding one output column per row as weights [out][in] do).  Integer products and sums are exact, and
// |acc| < 2^31 for k <= 65536, so every summation order gives the same int32: the k loop may be split,
// reordered and spread over matrix instructions freely.  The dequantised output is
// y[i][j] = RN(RN(RN32(acc) * sa) * sb[j]).
//
// Tiling: a workgroup of 4 wavefronts owns a 128 x 128 output tile, each wavefront a 64 x 64 block made of
// 2 x 2 v_mfma_i32_32x32x32_i8 blocks.  Stages of 64 k bytes are staged through LDS (rows padded to 80
// bytes, which makes the 16-byte operand reads of 32 consecutive rows conflict-free), double buffered.
// Each lane of a 32x32x32 instruction supplies 16 consecutive k bytes of one row of A and of B; the two
// half-wavefronts cover k 0..15 and 16..31 of the instruction's 32.
#include <hip/hip_runtime.h>

#include "canon_internal.h"

namespace canon {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));

constexpr int QBM = 128, QBN = 128, QKS = 64;
constexpr int QLD = QKS + 16;

struct I8Raw {
  uint4 a[2], b[2];
};

// 16 consecutive bytes of which the first `valid` exist (zero fill beyond)
template <bool FAST>
__device__ __forceinline__ uint4 ld16(const int8_t* p, int64_t valid, bool vec) {
  if (FAST || (vec && valid >= 16)) return *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  for (int e = 0; e < 16; ++e)
    if (e < valid) w[e >> 2] |= (uint32_t)(uint8_t)p[e] << (8 * (e & 3));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

template <bool FAST>
__device__ __forceinline__ I8Raw load_stage(const GemmI8Args& g, int64_t row0, int64_t col0, int64_t k0) {
  const int t = threadIdx.x;
  I8Raw r;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int idx = t + 256 * it;
    const int rr = idx >> 2;
    const int64_t k = k0 + 16 * (idx & 3);
    const int64_t row = row0 + rr, col = col0 + rr;
    r.a[it] = ld16<FAST>(g.a + row * g.lda + k, (row < g.m) ? g.k - k : 0, g.vec);
    r.b[it] = ld16<FAST>(g.b + col * g.ldb + k, (col < g.n) ? g.k - k : 0, g.vec);
  }
  return r;
}

__device__ __forceinline__ void store_stage(int8_t* As, int8_t* Bs, const I8Raw& r) {
  const int t = threadIdx.x;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int idx = t + 256 * it;
    const int off = (idx >> 2) * QLD + 16 * (idx & 3);
    *reinterpret_cast<uint4*>(As + off) = r.a[it];
    *reinterpret_cast<uint4*>(Bs + off) = r.b[it];
  }
}

__global__ __launch_bounds__(256) void gemm_i8_kernel(GemmI8Args g) {
  __shared__ __attribute__((aligned(16))) int8_t As[2][QBM * QLD];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][QBN * QLD];

  // tile order: a contiguous run of tiles per XCD, walked in groups of 8 tile rows
  constexpr int64_t GM = 8;
  const int64_t tiles_n = (g.n + QBN - 1) / QBN;
  const int64_t tiles_m = (g.m + QBM - 1) / QBM;
  const int64_t tiles = tiles_m * tiles_n;
  int64_t tile = blockIdx.x;
  if ((tiles & 7) == 0) tile = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int64_t group = tile / (GM * tiles_n);
  const int64_t first_m = group * GM;
  const int64_t gsize = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
  const int64_t within = tile - group * GM * tiles_n;
  const int64_t row0 = (first_m + within % gsize) * QBM, col0 = (within / gsize) * QBN;
  const bool tile_in = g.vec && row0 + QBM <= g.m && col0 + QBN <= g.n;

  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int ar = 64 * wr + (lane & 31), bc = 64 * wc + (lane & 31);
  const int kh = 16 * (lane >> 5);

  i32x16 acc[2][2];
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int v2 = 0; v2 < 2; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[h][v2][v] = 0;

  const int64_t ns = (g.k + QKS - 1) / QKS;
  int buf = 0;
  if (ns > 0) store_stage(As[0], Bs[0], load_stage<false>(g, row0, col0, 0));
  __syncthreads();
  for (int64_t s = 0; s < ns; ++s) {
    const bool more = s + 1 < ns;
    I8Raw nxt;
    if (more) {
      if (tile_in && (s + 2) * QKS <= g.k) nxt = load_stage<true>(g, row0, col0, (s + 1) * QKS);
      else nxt = load_stage<false>(g, row0, col0, (s + 1) * QKS);
    }
    __builtin_amdgcn_sched_barrier(0);
    const int8_t* as = As[buf];
    const int8_t* bs = Bs[buf];
#pragma unroll
    for (int ks = 0; ks < QKS / 32; ++ks) {
      const int kk = 32 * ks + kh;
      const i32x4 a0 = *reinterpret_cast<const i32x4*>(as + ar * QLD + kk);
      const i32x4 a1 = *reinterpret_cast<const i32x4*>(as + (ar + 32) * QLD + kk);
      const i32x4 b0 = *reinterpret_cast<const i32x4*>(bs + bc * QLD + kk);
      const i32x4 b1 = *reinterpret_cast<const i32x4*>(bs + (bc + 32) * QLD + kk);
      acc[0][0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, b0, acc[0][0], 0, 0, 0);
      acc[0][1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a0, b1, acc[0][1], 0, 0, 0);
      acc[1][0] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a1, b0, acc[1][0], 0, 0, 0);
      acc[1][1] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a1, b1, acc[1][1], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (more) store_stage(As[buf ^ 1], Bs[buf ^ 1], nxt);
    __syncthreads();
    buf ^= 1;
  }

  // result layout: register v, lane l -> row (v % 4) + 4 (l / 32) + 8 (v / 4), column l % 32 of the block
  const float sa = g.y ? *g.sa : 0.0f;
#pragma unroll
  for (int h = 0; h < 2; ++h)
#pragma unroll
    for (int v2 = 0; v2 < 2; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t i = row0 + 64 * wr + 32 * h + (v & 3) + 4 * (lane >> 5) + 8 * (v >> 2);
        const int64_t j = col0 + 64 * wc + 32 * v2 + (lane & 31);
        if (i < g.m && j < g.n) {
          const int32_t a = acc[h][v2][v];
          if (g.acc) g.acc[i * g.ldc + j] = a;
          if (g.y) {
            const float af = (float)a;  // round to nearest even
            const float t = af * sa;
            g.y[i * g.ldc + j] = t * g.sb[j];
          }
        }
      }
}

hipError_t gemm_i8_launch(const GemmI8Args& gin, hipStream_t s) {
  if (gin.m == 0 || gin.n == 0) return hipSuccess;
  GemmI8Args g = gin;
  g.vec = ((uintptr_t)g.a & 15) == 0 && ((uintptr_t)g.b & 15) == 0 && g.lda % 16 == 0 && g.ldb % 16 == 0;
  const int64_t tiles = ((g.m + QBM - 1) / QBM) * ((g.n + QBN - 1) / QBN);
  hipLaunchKernelGGL(gemm_i8_kernel, dim3((unsigned)tiles), dim3(256), 0, s, g);
  return hipGetLastError();
}

}  // namespace canon
