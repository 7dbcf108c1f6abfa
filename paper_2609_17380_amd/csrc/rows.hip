// rows.hip - row-wise canonical reductions: RMSNorm (R3), causal softmax (R5), cross-entropy (R6) and the
// row pieces of the attention backward.
//
// Layout of every row reduction: the row's chunks of 32 are split into aligned power-of-two blocks of G
// chunks, one block per lane (or thread).  Each lane folds its block with a register binary-carry stack
// (a complete or left-filled subtree of the padded tree), then the lanes are folded across the wavefront or
// workgroup with the pass-through rule, which together give Algorithm 2 over the row's chunks.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

__device__ __forceinline__ float wave_max(float m) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) m = fmaxf(m, __shfl_xor(m, s, 64));
  return m;
}

// ---- W-wide loads and stores (W = 1, 4 or 8 consecutive elements; the caller guarantees alignment) ----
template <int W>
__device__ __forceinline__ void ldf(const float* p, float (&f)[W]) {
  if constexpr (W == 1) {
    f[0] = p[0];
  } else {
#pragma unroll
    for (int i = 0; i < W; i += 4) {
      const float4 v = *reinterpret_cast<const float4*>(p + i);
      f[i] = v.x; f[i + 1] = v.y; f[i + 2] = v.z; f[i + 3] = v.w;
    }
  }
}

template <int W>
__device__ __forceinline__ void ldb(const uint16_t* p, float (&f)[W]) {
  if constexpr (W == 1) {
    f[0] = bf16_to_f32(p[0]);
  } else if constexpr (W == 4) {
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    f[0] = bf16_to_f32((uint16_t)(u.x & 0xFFFFu)); f[1] = bf16_to_f32((uint16_t)(u.x >> 16));
    f[2] = bf16_to_f32((uint16_t)(u.y & 0xFFFFu)); f[3] = bf16_to_f32((uint16_t)(u.y >> 16));
  } else {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = bf16_to_f32((uint16_t)(w4[i] & 0xFFFFu));
      f[2 * i + 1] = bf16_to_f32((uint16_t)(w4[i] >> 16));
    }
  }
}

__device__ __forceinline__ void ldb8_regs(const uint4& u, float (&f)[8]) {
  const uint32_t w4[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = bf16_to_f32((uint16_t)(w4[i] & 0xFFFFu));
    f[2 * i + 1] = bf16_to_f32((uint16_t)(w4[i] >> 16));
  }
}

template <int W>
__device__ __forceinline__ void stb(uint16_t* p, const uint16_t (&h)[W]) {
  if constexpr (W == 1) {
    p[0] = h[0];
  } else if constexpr (W == 4) {
    *reinterpret_cast<uint2*>(p) = make_uint2((uint32_t)h[0] | ((uint32_t)h[1] << 16),
                                              (uint32_t)h[2] | ((uint32_t)h[3] << 16));
  } else {
    *reinterpret_cast<uint4*>(p) =
        make_uint4((uint32_t)h[0] | ((uint32_t)h[1] << 16), (uint32_t)h[2] | ((uint32_t)h[3] << 16),
                   (uint32_t)h[4] | ((uint32_t)h[5] << 16), (uint32_t)h[6] | ((uint32_t)h[7] << 16));
  }
}

template <int W>
__device__ __forceinline__ void stf(float* p, const float (&f)[W]) {
  if constexpr (W == 1) {
    p[0] = f[0];
  } else {
#pragma unroll
    for (int i = 0; i < W; i += 4) *reinterpret_cast<float4*>(p + i) = make_float4(f[i], f[i + 1], f[i + 2], f[i + 3]);
  }
}

// ------------------------------------------------------------------------------------------------
// Coalesced row reduction for one wavefront.  A segment of 64 chunks (2048 terms) is read coalesced (lane l
// takes terms 64W q + W l .. + W-1), staged in LDS as padded rows [chunk][33], and lane c then runs chunk
// c's chain sequentially from LDS; the chunk partials of all segments collect in `parts` and are folded by
// lane blocks + wave_fold (Algorithm 2).  term(j, f) evaluates terms j .. j+W-1 of the row into f (for
// W > 1 the row length is a multiple of W, so a vector is either wholly inside the row or wholly past it).
struct WaveStage {
  float t[64][33];
};

template <int W, class Term>
__device__ __forceinline__ void wave_segment_chunks(int64_t seg0, int64_t n, WaveStage& st, float* parts, Term term) {
  const int lane = threadIdx.x & 63;
  const int64_t nc = (n + kChunk - 1) / kChunk;
#pragma unroll 2
  for (int q = 0; q < 64 * kChunk / (64 * W); ++q) {
    const int local = 64 * W * q + W * lane;
    const int64_t j = seg0 + local;
    float f[W];
    if (j < n) {
      term(j, f);
    } else {
#pragma unroll
      for (int i = 0; i < W; ++i) f[i] = 0.0f;
    }
    float* dst = &st.t[local >> 5][local & 31];
#pragma unroll
    for (int i = 0; i < W; ++i) dst[i] = f[i];
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  const int64_t c = seg0 / kChunk + lane;
  if (c < nc) {
    const int64_t k1 = n - c * kChunk < kChunk ? n - c * kChunk : kChunk;
    float s = 0.0f;
    for (int i = 0; i < (int)k1; ++i) s = s + st.t[lane][i];
    parts[c] = s;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
}

// nz: terms at index >= nz are known to be +0 (masked); z0: so are the terms below z0.  Chunks made only of
// such terms have partial +0: those at or after nz, and those of whole staging segments below z0, are not
// staged.
// Algorithm 2 over the nc chunk partials of one row in parts[] (written and made visible by the caller):
// lane l folds the block of G consecutive partials it owns, then the lane results are folded across the
// wavefront.  Returns the row sum in every lane.
__device__ __forceinline__ float fold_parts(const float* parts, int64_t nc) {
  const int lane = threadIdx.x & 63;
  const int64_t G = block_chunks(nc, 64);
  const int64_t c0 = lane * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  for (int64_t c = c0; c < c1; ++c) f.push(parts[c]);
  float tot = wave_fold(f.result(), (int)((nc + G - 1) / G));
  return __shfl(tot, 0, 64);
}

template <int W, class Term>
__device__ __forceinline__ float wave_row_rsum(int64_t n, WaveStage& st, float* parts, Term term, int64_t nz,
                                               int64_t z0 = 0) {
  const int lane = threadIdx.x & 63;
  const int64_t nc = (n + kChunk - 1) / kChunk;
  const int64_t zseg = (z0 / (64 * kChunk)) * (64 * kChunk);
  for (int64_t c = lane; c < zseg / kChunk && c < nc; c += 64) parts[c] = 0.0f;
  for (int64_t seg0 = zseg; seg0 < n && seg0 < nz; seg0 += 64 * kChunk) wave_segment_chunks<W>(seg0, n, st, parts, term);
  for (int64_t c = (nz + kChunk - 1) / kChunk + lane; c < nc; c += 64) parts[c] = 0.0f;
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  return fold_parts(parts, nc);
}

constexpr int kMaxRowChunks = 64 * 16;  // rows up to 32768 terms in the wave kernels

// The wave kernels take 4 rows per workgroup, with parts[] as dynamic LDS of 4 x (chunks per row) floats.
static inline size_t wave_kernel_lds(int64_t cols) { return sizeof(float) * 4 * (size_t)((cols + kChunk - 1) / kChunk); }

// Register-resident rows (cols <= 2048, a multiple of 4, aligned): lane l holds terms 4l + 256q .. +3 of
// its row for q < 8, read from memory once.  The chunk chains still run one per lane over a padded LDS
// transpose of the row (the same staging layout as wave_segment_chunks), then fold across the wavefront.
constexpr int kRegQ = 8;  // float4 vectors per lane: 64 x 4 x 8 = 2048 terms
constexpr int64_t kRegCols = 64 * 4 * kRegQ;

// Chain of every chunk of one staged row (nc <= 64 chunks, n terms) and the fold: returns the row sum.
__device__ __forceinline__ float reg_row_sum(WaveStage& st, const float (&e)[kRegQ][4], int64_t n) {
  const int lane = threadIdx.x & 63;
  const int nc = (int)((n + kChunk - 1) / kChunk);
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int local = 256 * q + 4 * lane;
    if (local < n) {
      float* dst = &st.t[local >> 5][local & 31];
#pragma unroll
      for (int t = 0; t < 4; ++t) dst[t] = e[q][t];
    }
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  float p = 0.0f;
  if (lane < nc) {
    const int k1 = (int)(n - (int64_t)lane * kChunk < kChunk ? n - (int64_t)lane * kChunk : kChunk);
    for (int i = 0; i < k1; ++i) p = p + st.t[lane][i];
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  return __shfl(wave_fold(p, nc), 0, 64);
}

// RMSNorm forward: one wavefront per row, 4 rows per workgroup.
template <int W, bool F32>
__global__ __launch_bounds__(256) void rownorm_fwd_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                          const uint16_t* __restrict__ gain, float eps, float inv_d,
                                                          void* __restrict__ y, float* __restrict__ rstd) {
  __shared__ WaveStage st[4];
  extern __shared__ float dyn[];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t nc = (cols + kChunk - 1) / kChunk;
  const float* xr = x + row * cols;
  float ss = wave_row_rsum<W>(cols, st[w], dyn + w * nc, [&](int64_t j, float (&f)[W]) {
    ldf<W>(xr + j, f);
#pragma unroll
    for (int i = 0; i < W; ++i) f[i] = f[i] * f[i];
  }, cols);
  float ms = ss * inv_d;
  float var = ms + eps;
  float r = 1.0f / __builtin_sqrtf(var);
  if (lane == 0) rstd[row] = r;
  for (int64_t k = (int64_t)lane * W; k < cols; k += 64 * W) {
    float xv[W], gv[W];
    uint16_t h[W];
    ldf<W>(xr + k, xv);
    ldb<W>(gain + k, gv);
    float o[W];
#pragma unroll
    for (int i = 0; i < W; ++i) {
      float xn = xv[i] * r;
      o[i] = xn * gv[i];
      h[i] = f32_to_bf16(o[i]);
    }
    if (F32) stf<W>((float*)y + row * cols + k, o);
    else stb<W>((uint16_t*)y + row * cols + k, h);
  }
}

// RMSNorm backward (dx): one wavefront per row.
// res (optional): dx = RN(res + the norm's gradient), the residual addition; dxb (optional): bf16 copy of dx.
template <int W>
__global__ __launch_bounds__(256) void rownorm_bwd_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                          const uint16_t* __restrict__ gain,
                                                          const float* __restrict__ rstd,
                                                          const float* __restrict__ dy, float inv_d,
                                                          float* __restrict__ dx, const float* __restrict__ res,
                                                          uint16_t* __restrict__ dxb) {
  __shared__ WaveStage st[4];
  extern __shared__ float dyn[];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t nc = (cols + kChunk - 1) / kChunk;
  const float* xr = x + row * cols;
  const float* dyr = dy + row * cols;
  float dot = wave_row_rsum<W>(cols, st[w], dyn + w * nc, [&](int64_t j, float (&f)[W]) {
    float dv[W], gv[W], xv[W];
    ldf<W>(dyr + j, dv);
    ldb<W>(gain + j, gv);
    ldf<W>(xr + j, xv);
#pragma unroll
    for (int i = 0; i < W; ++i) {
      float gy = dv[i] * gv[i];
      f[i] = gy * xv[i];
    }
  }, cols);
  const float r = rstd[row];
  float r2 = r * r;
  float r3 = r2 * r;
  float dd = dot * inv_d;
  float q = r3 * dd;
  for (int64_t k = (int64_t)lane * W; k < cols; k += 64 * W) {
    float dv[W], gv[W], xv[W], o[W];
    ldf<W>(dyr + k, dv);
    ldb<W>(gain + k, gv);
    ldf<W>(xr + k, xv);
#pragma unroll
    for (int i = 0; i < W; ++i) {
      float gy = dv[i] * gv[i];
      float a = r * gy;
      float b = xv[i] * q;
      o[i] = a - b;
    }
    if (res) {
      float rv[W];
      ldf<W>(res + row * cols + k, rv);
#pragma unroll
      for (int i = 0; i < W; ++i) o[i] = rv[i] + o[i];
    }
    stf<W>(dx + row * cols + k, o);
    if (dxb) {
      uint16_t h[W];
#pragma unroll
      for (int i = 0; i < W; ++i) h[i] = f32_to_bf16(o[i]);
      stb<W>(dxb + row * cols + k, h);
    }
  }
}

// RMSNorm forward and backward with register-resident rows (same arithmetic as the kernels above).
template <bool F32>
__global__ __launch_bounds__(256) void rownorm_fwd_reg_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                              const uint16_t* __restrict__ gain, float eps,
                                                              float inv_d, void* __restrict__ y,
                                                              float* __restrict__ rstd) {
  __shared__ WaveStage st[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const float* xr = x + row * cols;
  float xv[kRegQ][4], sq[kRegQ][4];
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    float v[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (j < cols) ldf<4>(xr + j, v);
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      xv[q][t] = v[t];
      sq[q][t] = v[t] * v[t];
    }
  }
  const float ss = reg_row_sum(st[w], sq, cols);
  float ms = ss * inv_d;
  float var = ms + eps;
  float r = 1.0f / __builtin_sqrtf(var);
  if (lane == 0) rstd[row] = r;
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    if (j < cols) {
      float gv[4], o[4];
      uint16_t h[4];
      ldb<4>(gain + j, gv);
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float xn = xv[q][t] * r;
        o[t] = xn * gv[t];
        h[t] = f32_to_bf16(o[t]);
      }
      if (F32) stf<4>((float*)y + row * cols + j, o);
      else stb<4>((uint16_t*)y + row * cols + j, h);
    }
  }
}

__global__ __launch_bounds__(256) void rownorm_bwd_reg_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                              const uint16_t* __restrict__ gain,
                                                              const float* __restrict__ rstd,
                                                              const float* __restrict__ dy, float inv_d,
                                                              float* __restrict__ dx, const float* __restrict__ res,
                                                              uint16_t* __restrict__ dxb) {
  __shared__ WaveStage st[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const float* xr = x + row * cols;
  const float* dyr = dy + row * cols;
  float xv[kRegQ][4], gy[kRegQ][4], tm[kRegQ][4];
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    float dv[4] = {0.0f, 0.0f, 0.0f, 0.0f}, gv[4] = {0.0f, 0.0f, 0.0f, 0.0f}, xx[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    if (j < cols) {
      ldf<4>(dyr + j, dv);
      ldb<4>(gain + j, gv);
      ldf<4>(xr + j, xx);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      xv[q][t] = xx[t];
      gy[q][t] = dv[t] * gv[t];
      tm[q][t] = gy[q][t] * xx[t];
    }
  }
  const float dot = reg_row_sum(st[w], tm, cols);
  const float r = rstd[row];
  float r2 = r * r;
  float r3 = r2 * r;
  float dd = dot * inv_d;
  float qq = r3 * dd;
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    if (j < cols) {
      float o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        float a = r * gy[q][t];
        float b = xv[q][t] * qq;
        o[t] = a - b;
      }
      if (res) {
        float rv[4];
        ldf<4>(res + row * cols + j, rv);
#pragma unroll
        for (int t = 0; t < 4; ++t) o[t] = rv[t] + o[t];
      }
      stf<4>(dx + row * cols + j, o);
      if (dxb) {
        uint16_t h[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) h[t] = f32_to_bf16(o[t]);
        stb<4>(dxb + row * cols + j, h);
      }
    }
  }
}

// dgain[k] = R1 over rows t of RN(dy[t,k] * RN(x[t,k] * rstd[t])), in two launches.  First every (chunk of
// 32 rows, column) chain, one per thread (lane = column, so row reads are coalesced), into part[c][k];
// then per column Algorithm 2 over its chunk partials in ascending order: a workgroup of 16 wavefronts
// takes 64 columns, wavefront q folds the aligned power-of-two group of chunks [q*G, q*G + G), and the 16
// group results are folded with the pass-through rule.
__global__ __launch_bounds__(256) void rownorm_dgain_part_kernel(int64_t rows, int64_t cols,
                                                                 const float* __restrict__ x,
                                                                 const float* __restrict__ rstd,
                                                                 const float* __restrict__ dy,
                                                                 float* __restrict__ part) {
  const int64_t col = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t c = blockIdx.y;
  if (col >= cols) return;
  const int64_t t0 = c * kChunk, t1 = (t0 + kChunk < rows) ? t0 + kChunk : rows;
  float s = 0.0f;
  for (int64_t t = t0; t < t1; ++t) {
    float xh = x[t * cols + col] * rstd[t];
    float pr = dy[t * cols + col] * xh;
    s = s + pr;
  }
  part[c * cols + col] = s;
}

constexpr int kDgainGroups = 16;
__global__ __launch_bounds__(1024) void rownorm_dgain_fold_kernel(int64_t rows, int64_t cols,
                                                                  const float* __restrict__ part,
                                                                  float* __restrict__ dgain) {
  __shared__ float gres[kDgainGroups][64];
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int64_t col = (int64_t)blockIdx.x * 64 + lane;
  const int64_t nc = (rows + kChunk - 1) / kChunk;
  const int64_t G = block_chunks(nc, kDgainGroups);
  const int64_t c0 = grp * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFoldN<22> f;
  if (col < cols) {
    int64_t c = c0;
    for (; c + 4 <= c1; c += 4) {
      const float p0 = part[c * cols + col], p1 = part[(c + 1) * cols + col];
      const float p2 = part[(c + 2) * cols + col], p3 = part[(c + 3) * cols + col];
      f.push(p0); f.push(p1); f.push(p2); f.push(p3);
    }
    for (; c < c1; ++c) f.push(part[c * cols + col]);
  }
  gres[grp][lane] = f.result();
  __syncthreads();
  if (grp == 0 && col < cols) {
    // fold the group results: level by level, a node adds its right neighbour when that subtree is real
    float v[kDgainGroups];
#pragma unroll
    for (int q = 0; q < kDgainGroups; ++q) v[q] = gres[q][lane];
#pragma unroll
    for (int sdist = 1; sdist < kDgainGroups; sdist <<= 1)
#pragma unroll
      for (int q = 0; q + sdist < kDgainGroups; q += 2 * sdist)
        if ((q + sdist) * G < nc) v[q] = v[q] + v[q + sdist];
    dgain[col] = v[0];
  }
}

static inline bool al(const void* p, unsigned a) { return ((uintptr_t)p & (a - 1)) == 0; }

template <bool F32>
static hipError_t rownorm_fwd_any(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps,
                                  void* y, float* rstd, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const float inv_d = (float)(1.0 / (double)cols);  // RN32(1/cols), correctly rounded
  const dim3 grid((unsigned)((rows + 3) / 4));
  const size_t lds = wave_kernel_lds(cols);
  const unsigned ya = F32 ? 16 : 8;
  if (cols % 4 == 0 && cols <= kRegCols && al(x, 16) && al(gain, 8) && al(y, ya))
    hipLaunchKernelGGL(rownorm_fwd_reg_kernel<F32>, grid, dim3(256), 0, s, rows, cols, x, gain, eps, inv_d, y, rstd);
  else if (cols % 4 == 0 && al(x, 16) && al(gain, 8) && al(y, ya))
    hipLaunchKernelGGL((rownorm_fwd_kernel<4, F32>), grid, dim3(256), lds, s, rows, cols, x, gain, eps, inv_d, y,
                       rstd);
  else
    hipLaunchKernelGGL((rownorm_fwd_kernel<1, F32>), grid, dim3(256), lds, s, rows, cols, x, gain, eps, inv_d, y,
                       rstd);
  return hipGetLastError();
}

hipError_t rownorm_fwd_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps, uint16_t* y,
                              float* rstd, hipStream_t s) {
  return rownorm_fwd_any<false>(rows, cols, x, gain, eps, y, rstd, s);
}

hipError_t rownorm_fwd_f32_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps,
                                  float* y, float* rstd, hipStream_t s) {
  return rownorm_fwd_any<true>(rows, cols, x, gain, eps, y, rstd, s);
}

// dx doubles as the scratch of the dgain chunk partials (ceil(rows/32) x cols floats <= rows x cols), so
// the dgain launches run before the dx kernel overwrites it.
hipError_t rownorm_bwd_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, const float* rstd,
                              const float* dy, float* dx, float* dgain, hipStream_t s, const float* res,
                              uint16_t* dxb) {
  if (dgain && res && res == dx) return hipErrorInvalidValue;  // dx holds the dgain partials before res is read
  if (rows == 0) {
    if (dgain) return hipMemsetAsync(dgain, 0, sizeof(float) * cols, s);
    return hipSuccess;
  }
  const float inv_d = (float)(1.0 / (double)cols);
  if (dgain) {
    const int64_t nc = (rows + kChunk - 1) / kChunk;
    hipLaunchKernelGGL(rownorm_dgain_part_kernel, dim3((unsigned)((cols + 255) / 256), (unsigned)nc), dim3(256), 0,
                       s, rows, cols, x, rstd, dy, dx);
    hipLaunchKernelGGL(rownorm_dgain_fold_kernel, dim3((unsigned)((cols + 63) / 64)), dim3(1024), 0, s, rows, cols,
                       dx, dgain);
  }
  const dim3 grid((unsigned)((rows + 3) / 4));
  const size_t lds = wave_kernel_lds(cols);
  const bool v4 = cols % 4 == 0 && al(x, 16) && al(gain, 8) && al(dy, 16) && al(dx, 16) && (!res || al(res, 16)) &&
                  (!dxb || al(dxb, 8));
  if (v4 && cols <= kRegCols)
    hipLaunchKernelGGL(rownorm_bwd_reg_kernel, grid, dim3(256), 0, s, rows, cols, x, gain, rstd, dy, inv_d, dx, res,
                       dxb);
  else if (v4)
    hipLaunchKernelGGL(rownorm_bwd_kernel<4>, grid, dim3(256), lds, s, rows, cols, x, gain, rstd, dy, inv_d, dx, res,
                       dxb);
  else
    hipLaunchKernelGGL(rownorm_bwd_kernel<1>, grid, dim3(256), lds, s, rows, cols, x, gain, rstd, dy, inv_d, dx, res,
                       dxb);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// LSQ step re-pin of the int8 quantised linear: per row r of a bf16 matrix,
// s[r] = RN(RN(2 * RN(R1(|w[r,:]|) * RN(1/cols))) * RN32(1/sqrt(127))).  One wavefront per row.
constexpr uint32_t kInvSqrtQmaxBits = 0x3DB5BB09u;  // RN32(1/sqrt(127))

template <int W>
__global__ __launch_bounds__(256) void quant_scales_kernel(int64_t rows, int64_t cols, const uint16_t* __restrict__ w,
                                                           float inv_k, float* __restrict__ scale) {
  __shared__ WaveStage st[4];
  extern __shared__ float dyn[];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wv;
  if (row >= rows) return;
  const int64_t nc = (cols + kChunk - 1) / kChunk;
  const uint16_t* wr = w + row * cols;
  const float a = wave_row_rsum<W>(cols, st[wv], dyn + wv * nc, [&](int64_t j, float (&f)[W]) {
    ldb<W>(wr + j, f);
#pragma unroll
    for (int i = 0; i < W; ++i) f[i] = __builtin_fabsf(f[i]);
  }, cols);
  const float mean = a * inv_k;
  const float two = 2.0f * mean;
  if (lane == 0) scale[row] = two * __uint_as_float(kInvSqrtQmaxBits);
}

// The same for rows held in registers (cols <= 2048, a multiple of 4, 8-byte aligned rows): one read of the row
__global__ __launch_bounds__(256) void quant_scales_reg_kernel(int64_t rows, int64_t cols,
                                                               const uint16_t* __restrict__ w, float inv_k,
                                                               float* __restrict__ scale) {
  __shared__ WaveStage st[4];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + wv;
  if (row >= rows) return;
  const uint16_t* wr = w + row * cols;
  float e[kRegQ][4];
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    if (j < cols) {
      float f[4];
      ldb<4>(wr + j, f);
#pragma unroll
      for (int t = 0; t < 4; ++t) e[q][t] = __builtin_fabsf(f[t]);
    } else {
#pragma unroll
      for (int t = 0; t < 4; ++t) e[q][t] = 0.0f;
    }
  }
  const float a = reg_row_sum(st[wv], e, cols);
  const float mean = a * inv_k;
  const float two = 2.0f * mean;
  if (lane == 0) scale[row] = two * __uint_as_float(kInvSqrtQmaxBits);
}

hipError_t quant_scales_launch(int64_t rows, int64_t cols, const uint16_t* w, float* scale, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const float inv_k = (float)(1.0 / (double)cols);  // RN32(1/cols)
  const dim3 grid((unsigned)((rows + 3) / 4));
  const size_t lds = wave_kernel_lds(cols);
  if (cols % 4 == 0 && cols <= kRegCols && al(w, 8))
    hipLaunchKernelGGL(quant_scales_reg_kernel, grid, dim3(256), 0, s, rows, cols, w, inv_k, scale);
  else if (cols % 4 == 0 && al(w, 8))
    hipLaunchKernelGGL(quant_scales_kernel<4>, grid, dim3(256), lds, s, rows, cols, w, inv_k, scale);
  else
    hipLaunchKernelGGL(quant_scales_kernel<1>, grid, dim3(256), lds, s, rows, cols, w, inv_k, scale);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// Causal softmax of raw scores: row r is query i = r mod cols; one wavefront per row, coalesced.  With
// window > 0 query i sees keys j0 = max(0, i - window + 1) .. i (the hybrid attention's windowed layers).
// band = 1 writes only the columns [wlo, whi) that the causally skipping products read (kAttnLead).
__device__ __forceinline__ void band_cols(int band, int64_t i, int64_t window, int64_t cols, int64_t& wlo,
                                          int64_t& whi) {
  if (!band) return;
  const int64_t lo = i - window - kAttnLead, hi = (i / 128) * 128 + 128;
  wlo = (window > 0 && lo > 0) ? lo : 0;
  whi = hi < cols ? hi : cols;
}
template <int W>
__global__ __launch_bounds__(256) void softmax_causal_kernel(int64_t rows, int64_t cols, const float* __restrict__ raw,
                                                             float scale, int64_t window,
                                                             uint16_t* __restrict__ probs, int band) {
  __shared__ WaveStage st[4];
  extern __shared__ float dyn[];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t nc = (cols + kChunk - 1) / kChunk;
  const int64_t i = row % cols;
  const int64_t j0 = (window > 0 && i - window + 1 > 0) ? i - window + 1 : 0;
  const float* rr = raw + row * cols;
  float m = -__builtin_inff();
  // keys before the window are not read: whole wavefront strides below j0 are skipped, and the loads of
  // vectors wholly below j0 are left out (their terms are +0 either way)
  for (int64_t j = (j0 / (64 * W)) * (64 * W) + (int64_t)lane * W; j <= i; j += 64 * W) {
    float v[W];
    ldf<W>(rr + j, v);
#pragma unroll
    for (int t = 0; t < W; ++t)
      if ((j + t <= i && j + t >= j0)) m = fmaxf(m, v[t] * scale);
  }
  m = wave_max(m);
  // masked keys enter the chain as +0 terms
  const float S = wave_row_rsum<W>(cols, st[w], dyn + w * nc, [&](int64_t j, float (&f)[W]) {
    float v[W];
    if (j + W - 1 >= j0) ldf<W>(rr + j, v);
#pragma unroll
    for (int t = 0; t < W; ++t) {
      float e = 0.0f;
      if ((j + t <= i && j + t >= j0)) {
        float sc = v[t] * scale;
        e = cexp(sc - m);
      }
      f[t] = e;
    }
  }, i + 1, j0);
  const float rcp = 1.0f / S;
  int64_t wlo = 0, whi = cols;  // columns written
  band_cols(band, i, window, cols, wlo, whi);
  for (int64_t j = (wlo / (64 * W)) * (64 * W) + (int64_t)lane * W; j < whi; j += 64 * W) {
    uint16_t o[W];
    if (j <= i && j + W - 1 >= j0) {
      float v[W];
      ldf<W>(rr + j, v);
#pragma unroll
      for (int t = 0; t < W; ++t) {
        o[t] = 0;
        if ((j + t <= i && j + t >= j0)) {
          float sc = v[t] * scale;
          float e = cexp(sc - m);
          o[t] = f32_to_bf16(e * rcp);
        }
      }
    } else {
#pragma unroll
      for (int t = 0; t < W; ++t) o[t] = 0;
    }
    stb<W>(probs + row * cols + j, o);
  }
}

__global__ __launch_bounds__(256) void softmax_causal_reg_kernel(int64_t rows, int64_t cols,
                                                                 const float* __restrict__ raw, float scale,
                                                                 int64_t window, uint16_t* __restrict__ probs,
                                                                 int band) {
  __shared__ WaveStage st[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t i = row % cols;
  const int64_t j0 = (window > 0 && i - window + 1 > 0) ? i - window + 1 : 0;
  const float* rr = raw + row * cols;
  float e[kRegQ][4];
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (j < cols && j <= i && j + 3 >= j0) v = *reinterpret_cast<const float4*>(rr + j);
    e[q][0] = v.x; e[q][1] = v.y; e[q][2] = v.z; e[q][3] = v.w;
  }
  float m = -__builtin_inff();
#pragma unroll
  for (int q = 0; q < kRegQ; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t j = 256 * q + 4 * lane + t;
      if (j < cols && j <= i && j >= j0) m = fmaxf(m, e[q][t] * scale);
    }
  m = wave_max(m);
  // masked keys enter the chain as +0 terms
#pragma unroll
  for (int q = 0; q < kRegQ; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int64_t j = 256 * q + 4 * lane + t;
      float x = 0.0f;
      if (j < cols && j <= i && j >= j0) {
        float sc = e[q][t] * scale;
        x = cexp(sc - m);
      }
      e[q][t] = x;
    }
  const float S = reg_row_sum(st[w], e, cols);
  const float rcp = 1.0f / S;
  int64_t wlo = 0, whi = cols;  // columns written
  band_cols(band, i, window, cols, wlo, whi);
#pragma unroll
  for (int q = 0; q < kRegQ; ++q) {
    const int64_t j = 256 * q + 4 * lane;
    if (j < whi && j + 3 >= wlo) {
      uint16_t o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) o[t] = ((j + t <= i && j + t >= j0)) ? f32_to_bf16(e[q][t] * rcp) : (uint16_t)0;
      stb<4>(probs + row * cols + j, o);
    }
  }
}

// Rows of 2048 < cols <= 4096 terms held in registers (lane l: terms 4l + 256q .. +3 for q < 16), read from
// memory once.  The chains run in two halves of 64 chunks through the same padded LDS transpose as
// wave_segment_chunks (lane c: chunk c, then chunk 64 + c), and the nc partials are folded as in
// wave_row_rsum (fold_parts).
constexpr int kReg2Q = 16;
constexpr int64_t kReg2Cols = 64 * 4 * kReg2Q;
__global__ __launch_bounds__(256) void softmax_causal_reg2_kernel(int64_t rows, int64_t cols,
                                                                  const float* __restrict__ raw, float scale,
                                                                  int64_t window, uint16_t* __restrict__ probs,
                                                                  int band) {
  __shared__ WaveStage st[4];
  extern __shared__ float dyn[];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t nc = (cols + kChunk - 1) / kChunk;
  float* parts = dyn + w * nc;
  const int i = (int)(row % cols);  // cols <= 4096: column indices fit in int
  const int j0 = (window > 0 && i - window + 1 > 0) ? (int)(i - window + 1) : 0;
  const int ncol = (int)cols;
  const float* rr = raw + row * cols;
  float e[kReg2Q][4];
#pragma unroll
  for (int q = 0; q < kReg2Q; ++q) {
    const int j = 256 * q + 4 * lane;
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (j < ncol && j <= i && j + 3 >= j0) v = *reinterpret_cast<const float4*>(rr + j);
    e[q][0] = v.x; e[q][1] = v.y; e[q][2] = v.z; e[q][3] = v.w;
  }
  float m = -__builtin_inff();
#pragma unroll
  for (int q = 0; q < kReg2Q; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = 256 * q + 4 * lane + t;
      if (j < ncol && j <= i && j >= j0) m = fmaxf(m, e[q][t] * scale);
    }
  m = wave_max(m);
  // masked keys enter the chain as +0 terms
#pragma unroll
  for (int q = 0; q < kReg2Q; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int j = 256 * q + 4 * lane + t;
      float x = 0.0f;
      if (j < ncol && j <= i && j >= j0) {
        float sc = e[q][t] * scale;
        x = cexp(sc - m);
      }
      e[q][t] = x;
    }
#pragma unroll
  for (int half = 0; half < 2; ++half) {
#pragma unroll
    for (int q = 0; q < kReg2Q / 2; ++q) {
      const int local = 256 * q + 4 * lane;
      if (2048 * half + local < ncol) {
        float* dst = &st[w].t[local >> 5][local & 31];
#pragma unroll
        for (int t = 0; t < 4; ++t) dst[t] = e[q + (kReg2Q / 2) * half][t];
      }
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
    const int c = 64 * half + lane;
    if (c < nc) {
      const int k1 = ncol - c * (int)kChunk < (int)kChunk ? ncol - c * (int)kChunk : (int)kChunk;
      float p = 0.0f;
      for (int k = 0; k < k1; ++k) p = p + st[w].t[lane][k];
      parts[c] = p;
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
  }
  const float S = fold_parts(parts, nc);
  const float rcp = 1.0f / S;
  int64_t wlo = 0, whi = cols;  // columns written
  band_cols(band, i, window, cols, wlo, whi);
#pragma unroll
  for (int q = 0; q < kReg2Q; ++q) {
    const int j = 256 * q + 4 * lane;
    if (j < whi && j + 3 >= wlo) {
      uint16_t o[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) o[t] = ((j + t <= i && j + t >= j0)) ? f32_to_bf16(e[q][t] * rcp) : (uint16_t)0;
      stb<4>(probs + row * cols + j, o);
    }
  }
}

// Windowed rows (0 < window <= kBandWin): the visible keys j0 .. i lie in the 768 columns [base, base + 768),
// base = j0 rounded down to 256, which lane l holds as float4 vectors at base + 256 q + 4 l (q < 3): the row
// is read from memory once.  The band's 24 chunks are staged in LDS and chained by lanes 0 .. 23 (every
// other chunk of the row is a +0 partial), and the nc partials are folded as in wave_row_rsum.
constexpr int64_t kBandWin = 512;
struct BandStage {
  float t[24][33];
};
__global__ __launch_bounds__(256) void softmax_band_kernel(int64_t rows, int64_t cols, const float* __restrict__ raw,
                                                           float scale, int64_t window, uint16_t* __restrict__ probs,
                                                           int band) {
  __shared__ BandStage st[4];
  extern __shared__ float dyn[];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t nc = (cols + kChunk - 1) / kChunk;
  float* parts = dyn + w * nc;
  const int64_t i = row % cols;
  const int64_t j0 = (i - window + 1 > 0) ? i - window + 1 : 0;
  const int64_t base = (j0 / 256) * 256;
  const float* rr = raw + row * cols;
  auto seen = [&](int64_t j) { return j <= i && j >= j0; };
  float e[3][4];
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const int64_t j = base + 256 * q + 4 * lane;
    float4 v = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (j < cols && j <= i && j + 3 >= j0) v = *reinterpret_cast<const float4*>(rr + j);
    e[q][0] = v.x; e[q][1] = v.y; e[q][2] = v.z; e[q][3] = v.w;
  }
  float m = -__builtin_inff();
#pragma unroll
  for (int q = 0; q < 3; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t)
      if (seen(base + 256 * q + 4 * lane + t)) m = fmaxf(m, e[q][t] * scale);
  m = wave_max(m);
  // masked keys enter the chain as +0 terms
#pragma unroll
  for (int q = 0; q < 3; ++q)
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      float x = 0.0f;
      if (seen(base + 256 * q + 4 * lane + t)) {
        float sc = e[q][t] * scale;
        x = cexp(sc - m);
      }
      e[q][t] = x;
    }
#pragma unroll
  for (int q = 0; q < 3; ++q) {
    const int local = 256 * q + 4 * lane;
    float* dst = &st[w].t[local >> 5][local & 31];
#pragma unroll
    for (int t = 0; t < 4; ++t) dst[t] = e[q][t];
  }
  for (int64_t c = lane; c < nc; c += 64) parts[c] = 0.0f;
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  const int64_t cb = base / kChunk + lane;  // this lane's band chunk
  if (lane < 24 && cb < nc) {
    const int64_t k1 = cols - cb * kChunk < kChunk ? cols - cb * kChunk : kChunk;
    float p = 0.0f;
    for (int k = 0; k < (int)k1; ++k) p = p + st[w].t[lane][k];
    parts[cb] = p;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  const float S = fold_parts(parts, nc);
  const float rcp = 1.0f / S;
  int64_t wlo = 0, whi = cols;  // columns written
  band_cols(band, i, window, cols, wlo, whi);
  for (int64_t j = (wlo / 256) * 256 + 4 * lane; j < whi; j += 256) {
    uint16_t o[4] = {0, 0, 0, 0};
    const int64_t d = j - base;
    if (d >= 0 && d < 768) {
      const int q = (int)(d >> 8);
      float x[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) x[t] = q == 0 ? e[0][t] : (q == 1 ? e[1][t] : e[2][t]);
#pragma unroll
      for (int t = 0; t < 4; ++t) o[t] = seen(j + t) ? f32_to_bf16(x[t] * rcp) : (uint16_t)0;
    }
    stb<4>(probs + row * cols + j, o);
  }
}

hipError_t softmax_causal_launch(int64_t rows, int64_t cols, const float* raw, float scale, int64_t window,
                                 uint16_t* probs, hipStream_t s, int band) {
  if (rows == 0) return hipSuccess;
  const dim3 grid((unsigned)((rows + 3) / 4));
  const size_t lds = wave_kernel_lds(cols);
  if (window > 0 && window <= kBandWin && cols % 4 == 0 && al(raw, 16) && al(probs, 8))
    hipLaunchKernelGGL(softmax_band_kernel, grid, dim3(256), lds, s, rows, cols, raw, scale, window, probs, band);
  else if (cols % 4 == 0 && cols <= kRegCols && al(raw, 16) && al(probs, 8))
    hipLaunchKernelGGL(softmax_causal_reg_kernel, grid, dim3(256), 0, s, rows, cols, raw, scale, window, probs,
                       band);
  else if (cols % 4 == 0 && cols <= kReg2Cols && al(raw, 16) && al(probs, 8))
    hipLaunchKernelGGL(softmax_causal_reg2_kernel, grid, dim3(256), lds, s, rows, cols, raw, scale, window, probs,
                       band);
  else if (cols % 4 == 0 && al(raw, 16) && al(probs, 8))
    hipLaunchKernelGGL(softmax_causal_kernel<4>, grid, dim3(256), lds, s, rows, cols, raw, scale, window, probs,
                       band);
  else
    hipLaunchKernelGGL(softmax_causal_kernel<1>, grid, dim3(256), lds, s, rows, cols, raw, scale, window, probs,
                       band);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// Cross-entropy: one 256-thread workgroup per row.  The four wavefronts take the row's 2048-term segments
// round-robin and write the chunk partials; the partials are then folded across the workgroup.  With W = 8
// (vocab a multiple of 8, 16-byte aligned logits and dlogits) every logit load and dlogit store moves 8 bf16
// values per lane.  parts[] is dynamic LDS sized to the row's chunk count.

template <int W>
__global__ __launch_bounds__(256) void xent_kernel(int64_t rows, int64_t vocab, const uint16_t* __restrict__ logits,
                                                   const int32_t* __restrict__ targets, float inv_tokens,
                                                   float z_loss, float z2, uint16_t* __restrict__ dlogits,
                                                   float* __restrict__ row_loss) {
  __shared__ WaveStage st[4];
  extern __shared__ float parts[];
  __shared__ float red[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = blockIdx.x;
  const uint16_t* lr = logits + row * vocab;
  float m = -__builtin_inff();
  for (int64_t j = (int64_t)threadIdx.x * W; j < vocab; j += 256 * W) {
    float f[W];
    ldb<W>(lr + j, f);
#pragma unroll
    for (int i = 0; i < W; ++i) m = fmaxf(m, f[i]);
  }
  m = wave_max(m);
  if (lane == 0) red[w] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  for (int64_t seg0 = (int64_t)w * 64 * kChunk; seg0 < vocab; seg0 += 4 * 64 * kChunk)
    wave_segment_chunks<W>(seg0, vocab, st[w], parts, [&](int64_t j, float (&f)[W]) {
      ldb<W>(lr + j, f);
#pragma unroll
      for (int i = 0; i < W; ++i) f[i] = cexp(f[i] - m);
    });
  __syncthreads();
  const int64_t nc = (vocab + kChunk - 1) / kChunk;
  const int64_t G = block_chunks(nc, 256);
  const int64_t c0 = threadIdx.x * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  for (int64_t c = c0; c < c1; ++c) f.push(parts[c]);
  const float S = block_fold(f.result(), (nc + G - 1) / G);
  const int32_t y = targets[row];
  const bool valid = y >= 0 && y < vocab;
  // z-loss (weight z_loss, z2 = RN(2 z_loss)): the row loss gains RN(z_loss * RN(lse^2)) and every
  // probability is scaled by RN(1 + RN(z2 * lse)) before the target is subtracted
  const float lse = m + clog(S);
  const bool zl = z_loss != 0.0f;
  const float zt = z2 * lse;
  const float pscale = 1.0f + zt;
  if (threadIdx.x == 0) {
    float ce = lse - bf16_to_f32(lr[valid ? y : 0]);
    if (zl) {
      const float l2 = lse * lse;
      const float zterm = z_loss * l2;
      ce = ce + zterm;
    }
    row_loss[row] = valid ? ce : __builtin_nanf("");
  }
  const float rcp = 1.0f / S;
  if (dlogits) {
    for (int64_t j = (int64_t)threadIdx.x * W; j < vocab; j += 256 * W) {
      float fv[W];
      uint16_t h[W];
      ldb<W>(lr + j, fv);
#pragma unroll
      for (int i = 0; i < W; ++i) {
        float e = cexp(fv[i] - m);
        float pr = e * rcp;
        if (zl) pr = pr * pscale;
        float q = pr - ((j + i) == y ? 1.0f : 0.0f);
        h[i] = f32_to_bf16(q * inv_tokens);
      }
      stb<W>(dlogits + row * vocab + j, h);
    }
  }
}

// Cross-entropy with the row's bf16 logits held in registers (vocab <= 51200, a multiple of 8, aligned):
// thread t holds elements 8 (t + 256 q) .. +7 for q < kXentQ, read once.  Segment s of 2048 terms is
// exactly vector q = s of every thread, so the workgroup stages four segments at a time (one per
// wavefront buffer, thread t writing chunk t/4 at offset 8 (t % 4)), then wavefront w runs the chains of
// segment buffer w.
constexpr int kXentQ = 25;
constexpr int64_t kXentRegVocab = 256 * 8 * kXentQ;

__global__ __launch_bounds__(256) void xent_reg_kernel(int64_t rows, int64_t vocab,
                                                       const uint16_t* __restrict__ logits,
                                                       const int32_t* __restrict__ targets, float inv_tokens,
                                                       float z_loss, float z2, uint16_t* __restrict__ dlogits,
                                                       float* __restrict__ row_loss) {
  __shared__ WaveStage st[4];
  extern __shared__ float parts[];
  __shared__ float red[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63, t = threadIdx.x;
  const int64_t row = blockIdx.x;
  const uint16_t* lr = logits + row * vocab;
  const int64_t n8 = vocab >> 3;
  uint4 raw[kXentQ];
#pragma unroll
  for (int q = 0; q < kXentQ; ++q) {
    const int64_t j8 = t + 256 * q;
    raw[q] = (j8 < n8) ? reinterpret_cast<const uint4*>(lr)[j8] : make_uint4(0u, 0u, 0u, 0u);
  }
  float m = -__builtin_inff();
#pragma unroll
  for (int q = 0; q < kXentQ; ++q) {
    if (t + 256 * q < n8) {
      float f[8];
      ldb8_regs(raw[q], f);
#pragma unroll
      for (int i = 0; i < 8; ++i) m = fmaxf(m, f[i]);
    }
  }
  m = wave_max(m);
  if (lane == 0) red[w] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  const int64_t nc = (vocab + kChunk - 1) / kChunk;
  const int nseg = (int)((vocab + 2047) / 2048);
#pragma unroll
  for (int s0 = 0; s0 < kXentQ; s0 += 4) {
    if (s0 < nseg) {
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const int sg = s0 + b;
        if (sg < kXentQ && sg < nseg && t + 256 * sg < n8) {
          float f[8];
          ldb8_regs(raw[sg], f);
          float* dst = &st[b].t[t >> 2][8 * (t & 3)];
#pragma unroll
          for (int i = 0; i < 8; ++i) dst[i] = cexp(f[i] - m);
        }
      }
      __syncthreads();
      const int sg = s0 + w;
      if (sg < nseg) {
        const int64_t c = (int64_t)sg * 64 + lane;
        if (c < nc) {
          const int64_t k1 = vocab - c * kChunk < kChunk ? vocab - c * kChunk : kChunk;
          float sacc = 0.0f;
          for (int i = 0; i < (int)k1; ++i) sacc = sacc + st[w].t[lane][i];
          parts[c] = sacc;
        }
      }
      __syncthreads();
    }
  }
  const int64_t G = block_chunks(nc, 256);
  const int64_t c0 = threadIdx.x * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  for (int64_t c = c0; c < c1; ++c) f.push(parts[c]);
  const float S = block_fold(f.result(), (nc + G - 1) / G);
  const int32_t y = targets[row];
  const bool valid = y >= 0 && y < vocab;
  // z-loss (weight z_loss, z2 = RN(2 z_loss)): the row loss gains RN(z_loss * RN(lse^2)) and every
  // probability is scaled by RN(1 + RN(z2 * lse)) before the target is subtracted
  const float lse = m + clog(S);
  const bool zl = z_loss != 0.0f;
  const float zt = z2 * lse;
  const float pscale = 1.0f + zt;
  if (threadIdx.x == 0) {
    float ce = lse - bf16_to_f32(lr[valid ? y : 0]);
    if (zl) {
      const float l2 = lse * lse;
      const float zterm = z_loss * l2;
      ce = ce + zterm;
    }
    row_loss[row] = valid ? ce : __builtin_nanf("");
  }
  const float rcp = 1.0f / S;
  if (dlogits) {
#pragma unroll
    for (int q = 0; q < kXentQ; ++q) {
      const int64_t j8 = t + 256 * q;
      if (j8 < n8) {
        float fv[8];
        uint16_t h[8];
        ldb8_regs(raw[q], fv);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          float e = cexp(fv[i] - m);
          float pr = e * rcp;
          if (zl) pr = pr * pscale;
          float qd = pr - ((j8 * 8 + i) == y ? 1.0f : 0.0f);
          h[i] = f32_to_bf16(qd * inv_tokens);
        }
        stb<8>(dlogits + row * vocab + j8 * 8, h);
      }
    }
  }
}

// mean_loss = RN(R1(row_loss) * inv_tokens): one workgroup.
__global__ __launch_bounds__(256) void mean_loss_kernel(int64_t rows, const float* __restrict__ row_loss,
                                                        float inv_tokens, float* __restrict__ out) {
  const int64_t nc = (rows + kChunk - 1) / kChunk;
  const int64_t G = block_chunks(nc, 256);
  const int64_t c0 = threadIdx.x * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  for (int64_t c = c0; c < c1; ++c) {
    float s = 0.0f;
    const int64_t k1 = (c + 1) * kChunk < rows ? (c + 1) * kChunk : rows;
    for (int64_t t = c * kChunk; t < k1; ++t) s = s + row_loss[t];
    f.push(s);
  }
  const float S = block_fold(f.result(), (nc + G - 1) / G);
  if (threadIdx.x == 0) out[0] = S * inv_tokens;
}

hipError_t xent_launch(int64_t rows, int64_t vocab, const uint16_t* logits, const int32_t* targets, float inv_tokens,
                       float z_loss, uint16_t* dlogits, float* row_loss, float* mean_loss, hipStream_t s) {
  if (rows > 0) {
    const size_t lds = sizeof(float) * (size_t)((vocab + kChunk - 1) / kChunk);
    const float z2 = 2.0f * z_loss;  // exact
    if (vocab % 8 == 0 && vocab <= kXentRegVocab && al(logits, 16) && al(dlogits, 16))
      hipLaunchKernelGGL(xent_reg_kernel, dim3((unsigned)rows), dim3(256), lds, s, rows, vocab, logits, targets,
                         inv_tokens, z_loss, z2, dlogits, row_loss);
    else if (vocab % 8 == 0 && al(logits, 16) && al(dlogits, 16))
      hipLaunchKernelGGL(xent_kernel<8>, dim3((unsigned)rows), dim3(256), lds, s, rows, vocab, logits, targets,
                         inv_tokens, z_loss, z2, dlogits, row_loss);
    else
      hipLaunchKernelGGL(xent_kernel<1>, dim3((unsigned)rows), dim3(256), lds, s, rows, vocab, logits, targets,
                         inv_tokens, z_loss, z2, dlogits, row_loss);
  }
  if (mean_loss)
    hipLaunchKernelGGL(mean_loss_kernel, dim3(1), dim3(256), 0, s, rows, row_loss, inv_tokens, mean_loss);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// D[bh][i] = R1 over d of fma(dO[i,d], O[i,d]) (bf16 operands, [T, ld] layout, head h at column h*hd).
// A row takes a group of G lanes (G = the chunk count rounded up to a power of two): lane r of the group
// runs the chain of chunk r over its 32 columns (16-byte loads when aligned, so the lanes of a group read the
// row's consecutive 64-byte pieces), and the group's first lane folds the chunk partials with Algorithm 2.
template <int G>
__global__ __launch_bounds__(256) void attn_rowdot_kernel(int64_t B, int64_t H, int64_t S, int64_t hd,
                                                          const uint16_t* __restrict__ dO,
                                                          const uint16_t* __restrict__ O, int64_t ld, int vec,
                                                          float* __restrict__ D) {
  const int64_t tid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t row = tid / G;
  const int r = (int)(tid % G);
  const int lane = threadIdx.x & 63;
  const bool live = row < B * H * S;
  const int nch = (int)((hd + kChunk - 1) / kChunk);
  float p = 0.0f;
  if (live && r < nch) {
    const int64_t i = row % S, bh = row / S, b = bh / H, h = bh % H;
    const int64_t off = (b * S + i) * ld + h * hd + (int64_t)r * kChunk;
    const uint16_t* a = dO + off;
    const uint16_t* o = O + off;
    const int64_t n = hd - (int64_t)r * kChunk < kChunk ? hd - (int64_t)r * kChunk : kChunk;
    if (vec && n == kChunk) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint4 av = reinterpret_cast<const uint4*>(a)[q];
        const uint4 ov = reinterpret_cast<const uint4*>(o)[q];
        const uint32_t aw[4] = {av.x, av.y, av.z, av.w}, ow[4] = {ov.x, ov.y, ov.z, ov.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          p = __builtin_fmaf(__uint_as_float(aw[e] << 16), __uint_as_float(ow[e] << 16), p);
          p = __builtin_fmaf(__uint_as_float(aw[e] & 0xFFFF0000u), __uint_as_float(ow[e] & 0xFFFF0000u), p);
        }
      }
    } else {
      for (int64_t k = 0; k < n; ++k) p = __builtin_fmaf(bf16_to_f32(a[k]), bf16_to_f32(o[k]), p);
    }
  }
  float parts[G];
#pragma unroll
  for (int q = 0; q < G; ++q) parts[q] = __shfl(p, (lane & ~(G - 1)) + q, 64);
  if (live && r == 0) {
    LocalFold f;
    for (int q = 0; q < nch; ++q) f.push(parts[q]);
    D[row] = f.result();
  }
}

// head dims above 16 chunks: one thread per row, chunks in order
__global__ __launch_bounds__(256) void attn_rowdot_wide_kernel(int64_t B, int64_t H, int64_t S, int64_t hd,
                                                               const uint16_t* __restrict__ dO,
                                                               const uint16_t* __restrict__ O, int64_t ld,
                                                               float* __restrict__ D) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * H * S) return;
  const int64_t i = idx % S, bh = idx / S, b = bh / H, h = bh % H;
  const uint16_t* a = dO + (b * S + i) * ld + h * hd;
  const uint16_t* o = O + (b * S + i) * ld + h * hd;
  LocalFold f;
  for (int64_t c0 = 0; c0 < hd; c0 += kChunk) {
    float p = 0.0f;
    const int64_t c1 = c0 + kChunk < hd ? c0 + kChunk : hd;
    for (int64_t k = c0; k < c1; ++k) p = __builtin_fmaf(bf16_to_f32(a[k]), bf16_to_f32(o[k]), p);
    f.push(p);
  }
  D[idx] = f.result();
}

hipError_t attn_rowdot_launch(int64_t B, int64_t H, int64_t S, int64_t hd, const uint16_t* dO, const uint16_t* O,
                              int64_t ld, float* D, hipStream_t s) {
  const int64_t n = B * H * S;
  if (n == 0) return hipSuccess;
  const int64_t nch = (hd + kChunk - 1) / kChunk;
  if (nch > 16) {
    hipLaunchKernelGGL(attn_rowdot_wide_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, B, H, S, hd, dO,
                       O, ld, D);
    return hipGetLastError();
  }
  const int vec = ((uintptr_t)dO & 15) == 0 && ((uintptr_t)O & 15) == 0 && ld % 8 == 0 && hd % 8 == 0;
  auto go = [&](auto gc) {
    constexpr int G = decltype(gc)::value;
    const int64_t threads = n * G;
    hipLaunchKernelGGL(attn_rowdot_kernel<G>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, s, B, H, S, hd,
                       dO, O, ld, vec, D);
  };
  if (nch <= 1) go(std::integral_constant<int, 1>{});
  else if (nch <= 2) go(std::integral_constant<int, 2>{});
  else if (nch <= 4) go(std::integral_constant<int, 4>{});
  else if (nch <= 8) go(std::integral_constant<int, 8>{});
  else go(std::integral_constant<int, 16>{});
  return hipGetLastError();
}

}  // namespace canon
