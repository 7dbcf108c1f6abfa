// qlinear.hip - backward of the int8 quantised linear: the straight-through gradients dx = dy . W^ and
// dW = dy^T . X^, each run as an int8 GEMM after a Walsh-Hadamard rotation of both operands along the
// contraction dimension (blocks of 256, the Sylvester matrix scaled by 1/16), with per-tensor absmax
// steps for the rotated operands.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

constexpr uint32_t kInv127Bits = 0x3C010204u;  // RN32(1/127)

enum { SRC_F32 = 0, SRC_I8 = 1, SRC_BF16 = 2 };

// dst [C][R] = transpose of src [R][C]: SRC_I8 int8 codes dequantised as RN(step * q) with step scale[r]
// (per_row) or scale[0]; SRC_F32 fp32 copied; SRC_BF16 bf16 widened (exact).  64 x 64 tiles through LDS.
template <int SRC>
__global__ __launch_bounds__(256) void transpose_kernel(int64_t R, int64_t C, const void* __restrict__ src,
                                                        const float* __restrict__ scale, int32_t per_row,
                                                        float* __restrict__ dst) {
  __shared__ float t[64][65];
  const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
  const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
  for (int i = ty; i < 64; i += 4) {
    const int64_t r = r0 + i, c = c0 + tx;
    float v = 0.0f;
    if (r < R && c < C) {
      if (SRC == SRC_I8) {
        const float s = scale[per_row ? r : 0];
        v = s * (float)static_cast<const int8_t*>(src)[r * C + c];
      } else if (SRC == SRC_BF16) {
        v = bf16_to_f32(static_cast<const uint16_t*>(src)[r * C + c]);
      } else {
        v = static_cast<const float*>(src)[r * C + c];
      }
    }
    t[i][tx] = v;
  }
  __syncthreads();
  for (int i = ty; i < 64; i += 4) {
    const int64_t c = c0 + i, r = r0 + tx;
    if (c < C && r < R) dst[c * R + r] = t[tx][i];
  }
}

// Blockwise rotation of src (n values, blocks of 256).  Each wavefront rotates blocks in a grid-stride loop,
// lane l holding values 4l .. 4l+3: butterflies of strides 1 and 2 inside the lane, the others across lanes
// by xor shuffles.  BF16: src holds bf16 values (widened exactly on load).  FWHT_AMAX: amax = max over the
// bit patterns of |result| (an atomic max of non-negative patterns, which is order-free; one atomic per
// workgroup); FWHT_QUANT: the rotation quantised with the per-tensor step *step (the R13 quantiser) into q.
// The rotated values are computed twice (once per pass) and never stored.
enum { FWHT_AMAX = 1, FWHT_QUANT = 2 };
template <bool BF16, int MODE>
__global__ __launch_bounds__(256) void fwht_kernel(int64_t n, const void* src, int8_t* __restrict__ q,
                                                   const float* __restrict__ step, uint32_t* __restrict__ amax) {
  __shared__ uint32_t wmax[4];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  uint32_t m = 0;
  float sv = 0.0f, rs = 0.0f;
  bool recip = false;
  if (MODE == FWHT_QUANT) {
    sv = step_daz(step[0]);
    recip = recip_step_ok(sv);
    rs = recip ? 1.0f / sv : 0.0f;
  }
  auto qz = [&](float v) -> uint32_t { return (uint8_t)(recip ? quant_recip(v, sv, rs) : quant1(v, sv)); };
  for (int64_t blk = (int64_t)blockIdx.x * 4 + wv; blk * 256 < n; blk += (int64_t)gridDim.x * 4) {
    float v[4];
    if (BF16) {
      const uint2 h = reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(src) + blk * 256)[lane];
      v[0] = __uint_as_float(h.x << 16);
      v[1] = __uint_as_float(h.x & 0xFFFF0000u);
      v[2] = __uint_as_float(h.y << 16);
      v[3] = __uint_as_float(h.y & 0xFFFF0000u);
    } else {
      const float4 x = reinterpret_cast<const float4*>(static_cast<const float*>(src) + blk * 256)[lane];
      v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    }
    {  // stride 1: pairs (0,1), (2,3); stride 2: pairs (0,2), (1,3)
      float a = v[0], b = v[1];
      v[0] = a + b; v[1] = a - b;
      a = v[2]; b = v[3];
      v[2] = a + b; v[3] = a - b;
      a = v[0]; b = v[2];
      v[0] = a + b; v[2] = a - b;
      a = v[1]; b = v[3];
      v[1] = a + b; v[3] = a - b;
    }
#pragma unroll
    for (int h = 4; h < 256; h <<= 1) {
      const int mask = h >> 2;
      const bool upper = (lane & mask) != 0;
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const float o = __shfl_xor(v[t], mask, 64);
        v[t] = upper ? o - v[t] : v[t] + o;
      }
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      v[t] = v[t] * 0.0625f;
      const uint32_t u = __float_as_uint(v[t]) & 0x7FFFFFFFu;
      m = u > m ? u : m;
    }
    if (MODE == FWHT_QUANT)
      reinterpret_cast<uint32_t*>(q + blk * 256)[lane] = qz(v[0]) | (qz(v[1]) << 8) | (qz(v[2]) << 16) | (qz(v[3]) << 24);
  }
  if (MODE == FWHT_QUANT) return;
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const uint32_t o = __shfl_xor(m, s, 64);
    m = o > m ? o : m;
  }
  if (lane == 0) wmax[wv] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t t = wmax[0];
    for (int i = 1; i < 4; ++i) t = wmax[i] > t ? wmax[i] : t;
    if (t) atomicMax(amax, t);
  }
}

__global__ void qlin_zero_kernel(uint32_t* amax, int n) {
  if ((int)threadIdx.x < n) amax[threadIdx.x] = 0u;
}

// step = RN(amax * RN(1/127)) for each of n cells
__global__ void qlin_step_kernel(const uint32_t* __restrict__ amax, float* __restrict__ step, int n) {
  if ((int)threadIdx.x < n) step[threadIdx.x] = __uint_as_float(amax[threadIdx.x]) * __uint_as_float(kInv127Bits);
}

template <int MODE>
static hipError_t fwht_launch(int64_t n, const void* src, int bf16, int8_t* q, const float* step, uint32_t* amax,
                              hipStream_t s) {
  const int64_t blocks = n / 256;
  if (blocks == 0) return hipSuccess;
  const int64_t wgs = (blocks + 3) / 4;
  const dim3 grid((unsigned)(wgs < 4096 ? wgs : 4096));
  if (bf16) hipLaunchKernelGGL((fwht_kernel<true, MODE>), grid, dim3(256), 0, s, n, src, q, step, amax);
  else hipLaunchKernelGGL((fwht_kernel<false, MODE>), grid, dim3(256), 0, s, n, src, q, step, amax);
  return hipGetLastError();
}
// amax of the rotation of src, then (after the step is formed) its codes: the rotated values are never stored
static hipError_t fwht_amax(int64_t n, const void* src, int bf16, uint32_t* amax, hipStream_t s) {
  return fwht_launch<FWHT_AMAX>(n, src, bf16, nullptr, nullptr, amax, s);
}
static hipError_t fwht_quant(int64_t n, const void* src, int bf16, const float* step, int8_t* q, hipStream_t s) {
  return fwht_launch<FWHT_QUANT>(n, src, bf16, q, step, nullptr, s);
}

template <int SRC>
static hipError_t transpose_launch(int64_t R, int64_t C, const void* src, const float* scale, int per_row,
                                   float* dst, hipStream_t s) {
  const dim3 grid((unsigned)((C + 63) / 64), (unsigned)((R + 63) / 64));
  hipLaunchKernelGGL(transpose_kernel<SRC>, grid, dim3(256), 0, s, R, C, src, scale, per_row, dst);
  return hipGetLastError();
}

size_t qlinear_bwd_workspace_bytes(int64_t T, int64_t N, int64_t K) {
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t big = (size_t)T * (size_t)N;
  const size_t small = (size_t)K * (size_t)(N > T ? N : T);
  return up(4 * big) + up(4 * small) + up(big) + up(small) + 256;
}

#define QTRY(x)                                   \
  do {                                            \
    hipError_t e_ = (x);                          \
    if (e_ != hipSuccess) return e_;              \
  } while (0)

hipError_t qlinear_bwd_launch(int64_t T, int64_t N, int64_t K, const void* dy, int dy_bf16, const int8_t* qx,
                              const float* sx, const int8_t* qw, const float* sw, float* dx, float* dw, void* ws,
                              hipStream_t s) {
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t big = (size_t)T * (size_t)N;
  const size_t small = (size_t)K * (size_t)(N > T ? N : T);
  char* p = (char*)ws;
  float* fa = (float*)p; p += up(4 * big);
  float* fb = (float*)p; p += up(4 * small);
  int8_t* qa = (int8_t*)p; p += up(big);
  int8_t* qb = (int8_t*)p; p += up(small);
  uint32_t* amax = (uint32_t*)p;       // 4 cells
  float* step = (float*)(p + 64);      // 4 cells
  hipLaunchKernelGGL(qlin_zero_kernel, dim3(1), dim3(64), 0, s, amax, 4);
  QTRY(hipGetLastError());
  if (dx) {  // contraction over N
    QTRY(fwht_amax(T * N, dy, dy_bf16, amax + 0, s));                      // rot(dy) [T][N]
    QTRY(transpose_launch<SRC_I8>(N, K, qw, sw, 1, fb, s));                // W^ transposed [K][N]
    QTRY(fwht_amax(K * N, fb, 0, amax + 1, s));
    hipLaunchKernelGGL(qlin_step_kernel, dim3(1), dim3(64), 0, s, amax, step, 2);
    QTRY(hipGetLastError());
    QTRY(fwht_quant(T * N, dy, dy_bf16, step + 0, qa, s));
    QTRY(fwht_quant(K * N, fb, 0, step + 1, qb, s));
    GemmI8Args g{};
    g.a = qa; g.b = qb; g.y = dx; g.sa = step + 0; g.sb = step + 1; g.sb_scalar = 1;
    g.m = T; g.n = K; g.k = N; g.lda = N; g.ldb = N; g.ldc = K;
    QTRY(gemm_i8_launch(g, s));
  }
  if (dw) {  // contraction over T
    if (dy_bf16) QTRY(transpose_launch<SRC_BF16>(T, N, dy, nullptr, 0, fa, s));  // dy transposed [N][T]
    else QTRY(transpose_launch<SRC_F32>(T, N, dy, nullptr, 0, fa, s));
    QTRY(fwht_amax(N * T, fa, 0, amax + 2, s));
    QTRY(transpose_launch<SRC_I8>(T, K, qx, sx, 0, fb, s));                // X^ transposed [K][T]
    QTRY(fwht_amax(K * T, fb, 0, amax + 3, s));
    hipLaunchKernelGGL(qlin_step_kernel, dim3(1), dim3(64), 0, s, amax + 2, step + 2, 2);
    QTRY(hipGetLastError());
    QTRY(fwht_quant(N * T, fa, 0, step + 2, qa, s));
    QTRY(fwht_quant(K * T, fb, 0, step + 3, qb, s));
    GemmI8Args g{};
    g.a = qa; g.b = qb; g.y = dw; g.sa = step + 2; g.sb = step + 3; g.sb_scalar = 1;
    g.m = N; g.n = K; g.k = T; g.lda = T; g.ldb = T; g.ldc = K;
    QTRY(gemm_i8_launch(g, s));
  }
  return hipSuccess;
}

}  // namespace canon
