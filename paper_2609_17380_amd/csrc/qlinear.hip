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
// Each operand's absmax is an atomic maximum spread over this many cells (one workgroup's atomic goes to cell
// workgroup mod kAmaxCells), so that thousands of workgroups do not queue on one address.
constexpr int kAmaxCells = 64;

// The rotation of a block of 256 values: 8 butterfly stages of strides 1, 2, 4, ..., 128, each pair (i, i + h)
// becoming (v_i + v_{i+h}, v_i - v_{i+h}) in binary32, then every value times 1/16 (exact).  The kernels hold
// 16 values of a block per lane and 16 lanes (one DPP row) per block, so four stages run inside the lane and four
// across the row's lanes.  Across lanes the partner is fetched by DPP (row-local lane permutations on the vector
// ALU) and the new value is fma(s, v, partner) with s = +1 in the lower and -1 in the upper lane of the pair:
// s v is exact, so this is one rounding of partner + v or partner - v, the same value as the add or subtract.
enum { FWHT_AMAX = 1, FWHT_QUANT = 2 };

// the value of lane (lane ^ M) of the same 16-lane row, M in {1, 2, 4, 8}
template <int M>
__device__ __forceinline__ float row_xor(float v) {
  const int x = __float_as_int(v);
  int r;
  if (M == 1) r = __builtin_amdgcn_update_dpp(0, x, 0xB1, 0xF, 0xF, false);        // quad_perm [1,0,3,2]
  else if (M == 2) r = __builtin_amdgcn_update_dpp(0, x, 0x4E, 0xF, 0xF, false);   // quad_perm [2,3,0,1]
  else if (M == 8) r = __builtin_amdgcn_update_dpp(0, x, 0x128, 0xF, 0xF, false);  // row_ror 8
  else {  // lanes 0-3 and 8-11 of the row read lane + 4 (row_ror 12), lanes 4-7 and 12-15 read lane - 4 (row_ror 4)
    const int t = __builtin_amdgcn_update_dpp(x, x, 0x12C, 0xF, 0x5, false);
    r = __builtin_amdgcn_update_dpp(t, x, 0x124, 0xF, 0xA, false);
  }
  return __int_as_float(r);
}
// stage across lanes: the pair is (lane, lane ^ M), the lane with bit M set holding the upper element
template <int M>
__device__ __forceinline__ void stage_lanes(float (&v)[16], int lane) {
  const float sgn = (lane & M) ? -1.0f : 1.0f;
#pragma unroll
  for (int j = 0; j < 16; ++j) v[j] = __builtin_fmaf(sgn, v[j], row_xor<M>(v[j]));
}
// stage inside the lane: pairs (j, j + H) of the lane's 16 values
template <int H>
__device__ __forceinline__ void stage_regs(float (&v)[16]) {
#pragma unroll
  for (int j = 0; j < 16; ++j)
    if (!(j & H)) {
      const float a = v[j], b = v[j + H];
      v[j] = a + b;
      v[j + H] = a - b;
    }
}

// Blockwise rotation of src (n values, blocks of 256 consecutive values; n a multiple of 256).  Lane L of a
// 16-lane row holds elements 16 L .. 16 L + 15 of its block (64 contiguous bytes), so strides 1 .. 8 are inside
// the lane and 16 .. 128 across the row; a wavefront rotates four blocks at a time in a grid-stride loop.
// BF16: src holds bf16 values (widened exactly on load).  FWHT_AMAX: amax = max over the bit patterns of
// |result| (an atomic max of non-negative patterns, which is order-free; one atomic per workgroup); FWHT_QUANT:
// the rotation quantised with the per-tensor step *step (the R13 quantiser) into q, 16 codes per lane.  The
// rotated values are computed twice (once per pass) and never stored.
template <bool BF16, int MODE>
__global__ __launch_bounds__(256) void fwht_kernel(int64_t n, const void* src, int8_t* __restrict__ q,
                                                   const float* __restrict__ step, uint32_t* __restrict__ amax) {
  __shared__ uint32_t wmax[4];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6, L = lane & 15;
  uint32_t m = 0;
  float sv = 0.0f, rs = 0.0f;
  bool recip = false;
  if (MODE == FWHT_QUANT) {
    sv = step_daz(step[0]);
    recip = recip_step_ok(sv);
    rs = recip ? 1.0f / sv : 0.0f;
  }
  auto qz = [&](float v) -> uint32_t { return (uint8_t)(recip ? quant_recip(v, sv, rs) : quant1(v, sv)); };
  const int64_t nblk = n / 256;
  for (int64_t blk = ((int64_t)blockIdx.x * 4 + wv) * 4 + (lane >> 4); blk < nblk; blk += (int64_t)gridDim.x * 16) {
    float v[16];
    if (BF16) {
      const uint4* p = reinterpret_cast<const uint4*>(static_cast<const uint16_t*>(src) + blk * 256 + 16 * L);
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const uint4 h = p[c];
        const uint32_t w[4] = {h.x, h.y, h.z, h.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[8 * c + 2 * e] = __uint_as_float(w[e] << 16);
          v[8 * c + 2 * e + 1] = __uint_as_float(w[e] & 0xFFFF0000u);
        }
      }
    } else {
      const float4* p = reinterpret_cast<const float4*>(static_cast<const float*>(src) + blk * 256 + 16 * L);
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const float4 x = p[c];
        v[4 * c] = x.x; v[4 * c + 1] = x.y; v[4 * c + 2] = x.z; v[4 * c + 3] = x.w;
      }
    }
    stage_regs<1>(v);
    stage_regs<2>(v);
    stage_regs<4>(v);
    stage_regs<8>(v);
    stage_lanes<1>(v, lane);
    stage_lanes<2>(v, lane);
    stage_lanes<4>(v, lane);
    stage_lanes<8>(v, lane);
    uint32_t w[4] = {0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      v[j] = v[j] * 0.0625f;
      if (MODE == FWHT_QUANT) {
        w[j >> 2] |= qz(v[j]) << (8 * (j & 3));
      } else {
        const uint32_t u = __float_as_uint(v[j]) & 0x7FFFFFFFu;
        m = u > m ? u : m;
      }
    }
    if (MODE == FWHT_QUANT) reinterpret_cast<uint4*>(q + blk * 256)[L] = make_uint4(w[0], w[1], w[2], w[3]);
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
    if (t) atomicMax(amax + (blockIdx.x & (kAmaxCells - 1)), t);  // spread over the cells (order-free)
  }
}

// The same rotation along the rows of src [R][C] (R a multiple of 256): for every column, blocks of 256
// consecutive rows, i.e. the rotation of the transposed matrix without forming it.  Source values: SRC_I8 codes
// dequantised as RN(scale * q) with scale[r] (per_row) or scale[0]; SRC_BF16 widened (exact); SRC_F32 as is.
// A workgroup stages a 256 x 32 tile through LDS (8 lanes per row segment, each 4 columns, all loads in flight
// before the first store).  Lane L of a 16-lane row then holds rows L, L + 16, ..., L + 240 of one column, so
// strides 1 .. 8 run across the row's lanes and 16 .. 128 inside the lane (in that order, as in fwht_kernel);
// the two 16-lane rows of each half-wavefront take columns 16 apart, which keeps the LDS reads free of bank
// conflicts.  FWHT_AMAX: amax as in fwht_kernel; FWHT_QUANT: codes written transposed, q [C][R], staged in LDS
// so that each column's 256 codes leave as one 256-byte run.
template <int SRC, int MODE>
__global__ __launch_bounds__(256) void fwht_cols_kernel(int64_t R, int64_t C, const void* __restrict__ src,
                                                        const float* __restrict__ scale, int32_t per_row,
                                                        int8_t* __restrict__ q, const float* __restrict__ step,
                                                        uint32_t* __restrict__ amax, int32_t vec4) {
  constexpr int TC = 32, LDT = TC + 1;
  __shared__ float t[256 * LDT];
  __shared__ uint32_t wmax[4];
  const int64_t r0 = (int64_t)blockIdx.y * 256, c0 = (int64_t)blockIdx.x * TC;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  {
    const int g4 = 4 * (lane & 7), rr = 8 * wv + (lane >> 3);
    const int64_t c = c0 + g4;
    float v[8][4];
    if (vec4 && c0 + TC <= C) {  // the whole tile in range (workgroup-uniform): 4-element vector loads
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const int64_t r = r0 + rr + 32 * it;
        const int64_t o = r * C + c;
        if (SRC == SRC_F32) {
          const float4 x = *reinterpret_cast<const float4*>(static_cast<const float*>(src) + o);
          v[it][0] = x.x; v[it][1] = x.y; v[it][2] = x.z; v[it][3] = x.w;
        } else if (SRC == SRC_BF16) {
          const uint2 h = *reinterpret_cast<const uint2*>(static_cast<const uint16_t*>(src) + o);
          v[it][0] = __uint_as_float(h.x << 16); v[it][1] = __uint_as_float(h.x & 0xFFFF0000u);
          v[it][2] = __uint_as_float(h.y << 16); v[it][3] = __uint_as_float(h.y & 0xFFFF0000u);
        } else {
          const uint32_t b = *reinterpret_cast<const uint32_t*>(static_cast<const int8_t*>(src) + o);
          const float sc = scale[per_row ? r : 0];
#pragma unroll
          for (int e = 0; e < 4; ++e) v[it][e] = sc * (float)(int8_t)(b >> (8 * e));
        }
      }
    } else {  // a ragged last tile or unaligned rows: element by element, +0 beyond the last column
#pragma unroll
      for (int it = 0; it < 8; ++it) {
        const int64_t r = r0 + rr + 32 * it;
        const int64_t o = r * C + c;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          float x = 0.0f;
          if (c + e < C) {
            if (SRC == SRC_I8) x = scale[per_row ? r : 0] * (float)static_cast<const int8_t*>(src)[o + e];
            else if (SRC == SRC_BF16) x = bf16_to_f32(static_cast<const uint16_t*>(src)[o + e]);
            else x = static_cast<const float*>(src)[o + e];
          }
          v[it][e] = x;
        }
      }
    }
#pragma unroll
    for (int it = 0; it < 8; ++it)
#pragma unroll
      for (int e = 0; e < 4; ++e) t[(rr + 32 * it) * LDT + g4 + e] = v[it][e];
  }
  __syncthreads();
  float sv = 0.0f, rs = 0.0f;
  bool recip = false;
  if (MODE == FWHT_QUANT) {
    sv = step_daz(step[0]);
    recip = recip_step_ok(sv);
    rs = recip ? 1.0f / sv : 0.0f;
  }
  const int L = lane & 15, k = lane >> 4;
  uint32_t m = 0;
  uint32_t codes[2][4];  // pass p: the codes of rows L + 16 j, j = 0..15, four per word
#pragma unroll
  for (int p = 0; p < 2; ++p) {
    // columns: k = 0, 1 (lanes 0-31) 16 apart, k = 2, 3 likewise; the 4 waves x 2 passes x 4 rows cover 32
    const int cc = (k & 1) * 16 + (k >> 1) * 8 + 2 * wv + p;
    float v[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) v[j] = t[(L + 16 * j) * LDT + cc];
    stage_lanes<1>(v, lane);
    stage_lanes<2>(v, lane);
    stage_lanes<4>(v, lane);
    stage_lanes<8>(v, lane);
    stage_regs<1>(v);
    stage_regs<2>(v);
    stage_regs<4>(v);
    stage_regs<8>(v);
    codes[p][0] = codes[p][1] = codes[p][2] = codes[p][3] = 0u;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      v[j] = v[j] * 0.0625f;
      if (MODE == FWHT_QUANT) {
        codes[p][j >> 2] |= (uint32_t)(uint8_t)(recip ? quant_recip(v[j], sv, rs) : quant1(v[j], sv)) << (8 * (j & 3));
      } else {
        const uint32_t u = __float_as_uint(v[j]) & 0x7FFFFFFFu;
        m = u > m ? u : m;
      }
    }
  }
  if (MODE == FWHT_QUANT) {
    // codes through LDS (the value tile is no longer read once every wavefront passed the barrier):
    // byte (column cc, row i) at cc * 256 + i
    __syncthreads();
    uint8_t* qt = reinterpret_cast<uint8_t*>(t);
#pragma unroll
    for (int p = 0; p < 2; ++p) {
      const int cc = (k & 1) * 16 + (k >> 1) * 8 + 2 * wv + p;
#pragma unroll
      for (int j = 0; j < 16; ++j) qt[cc * 256 + L + 16 * j] = (uint8_t)(codes[p][j >> 2] >> (8 * (j & 3)));
    }
    __syncthreads();
    // 32 columns x 64 words: thread x writes words x, x + 256, ... (each column's 64 words contiguous)
    const uint32_t* qw = reinterpret_cast<const uint32_t*>(qt);
#pragma unroll
    for (int w = threadIdx.x; w < TC * 64; w += 256) {
      const int cc = w >> 6, word = w & 63;
      if (c0 + cc < C) reinterpret_cast<uint32_t*>(q + (c0 + cc) * R + r0)[word] = qw[w];
    }
    return;
  }
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) {
    const uint32_t o = __shfl_xor(m, s, 64);
    m = o > m ? o : m;
  }
  if (lane == 0) wmax[wv] = m;
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t x = wmax[0];
    for (int i = 1; i < 4; ++i) x = wmax[i] > x ? wmax[i] : x;
    if (x) atomicMax(amax + ((blockIdx.x + blockIdx.y * gridDim.x) & (kAmaxCells - 1)), x);  // spread (order-free)
  }
}

__global__ void qlin_zero_kernel(uint32_t* amax, int n) {
  for (int i = threadIdx.x; i < n * kAmaxCells; i += blockDim.x) amax[i] = 0u;
}

// step = RN(amax * RN(1/127)) for each of n operands, amax the largest of the operand's cells
__global__ void qlin_step_kernel(const uint32_t* __restrict__ amax, float* __restrict__ step, int n) {
  if ((int)threadIdx.x < n) {
    uint32_t m = 0;
    for (int c = 0; c < kAmaxCells; ++c) {
      const uint32_t x = amax[threadIdx.x * kAmaxCells + c];
      m = x > m ? x : m;
    }
    step[threadIdx.x] = __uint_as_float(m) * __uint_as_float(kInv127Bits);
  }
}

template <int MODE>
static hipError_t fwht_launch(int64_t n, const void* src, int bf16, int8_t* q, const float* step, uint32_t* amax,
                              hipStream_t s) {
  const int64_t blocks = n / 256;
  if (blocks == 0) return hipSuccess;
  const int64_t wgs = (blocks + 15) / 16;  // 16 blocks per workgroup per iteration
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

template <int SRC, int MODE>
static hipError_t fwht_cols_launch(int64_t R, int64_t C, const void* src, const float* scale, int per_row, int8_t* q,
                                   const float* step, uint32_t* amax, hipStream_t s) {
  if (R == 0 || C == 0) return hipSuccess;
  const dim3 grid((unsigned)((C + 31) / 32), (unsigned)(R / 256));
  const int esz = SRC == SRC_F32 ? 4 : SRC == SRC_BF16 ? 2 : 1;  // vector loads of 4 elements need alignment
  const int vec4 = C % 4 == 0 && ((uintptr_t)src % (4 * esz)) == 0;
  hipLaunchKernelGGL((fwht_cols_kernel<SRC, MODE>), grid, dim3(256), 0, s, R, C, src, scale, per_row, q, step, amax,
                     vec4);
  return hipGetLastError();
}

size_t qlinear_bwd_workspace_bytes(int64_t T, int64_t N, int64_t K) {
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t big = (size_t)T * (size_t)N;
  const size_t small = (size_t)K * (size_t)(N > T ? N : T);
  return up(big) + up(small) + up(4 * kAmaxCells * sizeof(uint32_t)) + 256;
}

#define QTRY(x)                                   \
  do {                                            \
    hipError_t e_ = (x);                          \
    if (e_ != hipSuccess) return e_;              \
  } while (0)

// Each operand is rotated twice without being stored: a pass for its absmax, then (once the step is formed)
// a pass that writes its codes, already laid out contraction-contiguous for the GEMM.
hipError_t qlinear_bwd_launch(int64_t T, int64_t N, int64_t K, const void* dy, int dy_bf16, const int8_t* qx,
                              const float* sx, const int8_t* qw, const float* sw, float* dx, float* dw, void* ws,
                              hipStream_t s) {
  auto up = [](size_t b) { return (b + 255) & ~(size_t)255; };
  const size_t big = (size_t)T * (size_t)N;
  const size_t small = (size_t)K * (size_t)(N > T ? N : T);
  char* p = (char*)ws;
  int8_t* qa = (int8_t*)p; p += up(big);
  int8_t* qb = (int8_t*)p; p += up(small);
  uint32_t* amax = (uint32_t*)p;                            // 4 operands x kAmaxCells cells
  float* step = (float*)(p + up(4 * kAmaxCells * sizeof(uint32_t)));  // 4 cells
  hipLaunchKernelGGL(qlin_zero_kernel, dim3(1), dim3(256), 0, s, amax, 4);
  QTRY(hipGetLastError());
  if (dx) {  // contraction over N: rot(dy) along its rows' N, rot(W^) along N, codes of W^ as [K][N]
    QTRY(fwht_amax(T * N, dy, dy_bf16, amax + 0 * kAmaxCells, s));
    QTRY((fwht_cols_launch<SRC_I8, FWHT_AMAX>(N, K, qw, sw, 1, nullptr, nullptr, amax + 1 * kAmaxCells, s)));
    hipLaunchKernelGGL(qlin_step_kernel, dim3(1), dim3(64), 0, s, amax, step, 2);
    QTRY(hipGetLastError());
    QTRY(fwht_quant(T * N, dy, dy_bf16, step + 0, qa, s));
    QTRY((fwht_cols_launch<SRC_I8, FWHT_QUANT>(N, K, qw, sw, 1, qb, step + 1, nullptr, s)));
    GemmI8Args g{};
    g.a = qa; g.b = qb; g.y = dx; g.sa = step + 0; g.sb = step + 1; g.sb_scalar = 1;
    g.m = T; g.n = K; g.k = N; g.lda = N; g.ldb = N; g.ldc = K;
    QTRY(gemm_i8_launch(g, s));
  }
  if (dw) {  // contraction over T: rot(dy) along T with codes as [N][T], rot(X^) along T with codes as [K][T]
    if (dy_bf16) QTRY((fwht_cols_launch<SRC_BF16, FWHT_AMAX>(T, N, dy, nullptr, 0, nullptr, nullptr, amax + 2 * kAmaxCells, s)));
    else QTRY((fwht_cols_launch<SRC_F32, FWHT_AMAX>(T, N, dy, nullptr, 0, nullptr, nullptr, amax + 2 * kAmaxCells, s)));
    QTRY((fwht_cols_launch<SRC_I8, FWHT_AMAX>(T, K, qx, sx, 0, nullptr, nullptr, amax + 3 * kAmaxCells, s)));
    hipLaunchKernelGGL(qlin_step_kernel, dim3(1), dim3(64), 0, s, amax + 2 * kAmaxCells, step + 2, 2);
    QTRY(hipGetLastError());
    if (dy_bf16) QTRY((fwht_cols_launch<SRC_BF16, FWHT_QUANT>(T, N, dy, nullptr, 0, qa, step + 2, nullptr, s)));
    else QTRY((fwht_cols_launch<SRC_F32, FWHT_QUANT>(T, N, dy, nullptr, 0, qa, step + 2, nullptr, s)));
    QTRY((fwht_cols_launch<SRC_I8, FWHT_QUANT>(T, K, qx, sx, 0, qb, step + 3, nullptr, s)));
    GemmI8Args g{};
    g.a = qa; g.b = qb; g.y = dw; g.sa = step + 2; g.sb = step + 3; g.sb_scalar = 1;
    g.m = N; g.n = K; g.k = T; g.lda = T; g.ldb = T; g.ldc = K;
    QTRY(gemm_i8_launch(g, s));
  }
  return hipSuccess;
}

}  // namespace canon
