// rows.hip - row-wise canonical reductions: RMSNorm (R3), causal softmax (R5), cross-entropy (R6) and the
// row pieces of the attention backward.
//
// Layout of every row reduction: the row's chunks of 32 are split into aligned power-of-two blocks of G
// chunks, one block per lane (or thread).  Each lane folds its block with a register binary-carry stack
// (a complete or left-filled subtree of the padded tree), then the lanes are folded across the wavefront or
// workgroup with the pass-through rule, which together give Algorithm 2 over the row's chunks.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

constexpr int kLocalLevels = 16;  // a lane block of up to 2^15 chunks

struct LocalFold {
  float s[kLocalLevels];
  int64_t count = 0;
  __device__ void push(float p) {
#pragma unroll
    for (int L = 0; L < kLocalLevels; ++L) {
      if ((count >> L) & 1) {
        p = s[L] + p;
      } else {
        s[L] = p;
        break;
      }
    }
    ++count;
  }
  __device__ float result() const {
    float r = 0.0f;
    bool have = false;
#pragma unroll
    for (int L = 0; L < kLocalLevels; ++L) {
      if ((count >> L) & 1) {
        if (!have) { r = s[L]; have = true; }
        else r = s[L] + r;
      }
    }
    return r;
  }
};

// chunks per lane so that `lanes` lanes cover nc chunks with aligned power-of-two blocks
__device__ __forceinline__ int64_t block_chunks(int64_t nc, int lanes) {
  int64_t G = 1;
  while (G * lanes < nc) G <<= 1;
  return G;
}

// Fold of per-thread partials across a 256-thread workgroup; thread t holds part t (valid for t < nparts).
// Returns the total to every thread.
__device__ float block_fold(float p, int64_t nparts) {
  __shared__ float wsum[4];
  __shared__ float total;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t nl = nparts - 64 * w;
  nl = nl < 0 ? 0 : (nl > 64 ? 64 : nl);
  float r = wave_fold(p, (int)nl);
  if (lane == 0) wsum[w] = r;
  __syncthreads();
  if (threadIdx.x == 0) {
    float a = wsum[0];
    if (64 < nparts) a = a + wsum[1];
    float b = wsum[2];
    if (192 < nparts) b = b + wsum[3];
    if (128 < nparts) a = a + b;
    total = a;
  }
  __syncthreads();
  float t = total;
  __syncthreads();
  return t;
}

__device__ __forceinline__ float wave_max(float m) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) m = fmaxf(m, __shfl_xor(m, s, 64));
  return m;
}

// ------------------------------------------------------------------------------------------------
// Coalesced row reduction for one wavefront.  A segment of 64 chunks (2048 terms) is read coalesced (lane l
// takes terms 64q + l), staged in LDS as padded rows [chunk][33], and lane c then runs chunk c's chain
// sequentially from LDS; the chunk partials of all segments collect in `parts` and are folded by lane
// blocks + wave_fold (Algorithm 2).  term(j) evaluates the j-th term of the row.
struct WaveStage {
  float t[64][33];
};

// Stage one segment (terms seg0 .. seg0 + 2047 of a row of n terms) and write its chunk partials to parts.
template <class Term>
__device__ __forceinline__ void wave_segment_chunks(int64_t seg0, int64_t n, WaveStage& st, float* parts, Term term) {
  const int lane = threadIdx.x & 63;
  const int64_t nc = (n + kChunk - 1) / kChunk;
#pragma unroll 4
  for (int q = 0; q < 32; ++q) {
    const int local = 64 * q + lane;
    const int64_t j = seg0 + local;
    st.t[local >> 5][local & 31] = (j < n) ? term(j) : 0.0f;
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

// nz: terms at index >= nz are known to be +0 (masked); chunks made only of them have partial +0 and are not
// staged.
template <class Term>
__device__ __forceinline__ float wave_row_rsum(int64_t n, WaveStage& st, float* parts, Term term, int64_t nz) {
  const int lane = threadIdx.x & 63;
  const int64_t nc = (n + kChunk - 1) / kChunk;
  for (int64_t seg0 = 0; seg0 < n && seg0 < nz; seg0 += 64 * kChunk) wave_segment_chunks(seg0, n, st, parts, term);
  for (int64_t c = (nz + kChunk - 1) / kChunk + lane; c < nc; c += 64) parts[c] = 0.0f;
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  const int64_t G = block_chunks(nc, 64);
  const int64_t c0 = lane * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  for (int64_t c = c0; c < c1; ++c) f.push(parts[c]);
  float tot = wave_fold(f.result(), (int)((nc + G - 1) / G));
  return __shfl(tot, 0, 64);
}

constexpr int kMaxRowChunks = 64 * 16;  // rows up to 32768 terms in the wave kernels

// RMSNorm forward: one wavefront per row, 4 rows per workgroup.
__global__ __launch_bounds__(256) void rownorm_fwd_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                          const uint16_t* __restrict__ gain, float eps, float inv_d,
                                                          uint16_t* __restrict__ y, float* __restrict__ rstd) {
  __shared__ WaveStage st[4];
  __shared__ float parts[4][kMaxRowChunks];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const float* xr = x + row * cols;
  float ss = wave_row_rsum(cols, st[w], parts[w], [&](int64_t j) {
    float v = xr[j];
    return v * v;
  }, cols);
  float ms = ss * inv_d;
  float var = ms + eps;
  float r = 1.0f / __builtin_sqrtf(var);
  if (lane == 0) rstd[row] = r;
  for (int64_t k = lane; k < cols; k += 64) {
    float xv = xr[k] * r;
    float yv = xv * bf16_to_f32(gain[k]);
    y[row * cols + k] = f32_to_bf16(yv);
  }
}

// RMSNorm backward (dx): one wavefront per row.
__global__ __launch_bounds__(256) void rownorm_bwd_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                          const uint16_t* __restrict__ gain,
                                                          const float* __restrict__ rstd,
                                                          const float* __restrict__ dy, float inv_d,
                                                          float* __restrict__ dx) {
  __shared__ WaveStage st[4];
  __shared__ float parts[4][kMaxRowChunks];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const float* xr = x + row * cols;
  const float* dyr = dy + row * cols;
  float dot = wave_row_rsum(cols, st[w], parts[w], [&](int64_t j) {
    float gy = dyr[j] * bf16_to_f32(gain[j]);
    return gy * xr[j];
  }, cols);
  const float r = rstd[row];
  float r2 = r * r;
  float r3 = r2 * r;
  float dd = dot * inv_d;
  float q = r3 * dd;
  for (int64_t k = lane; k < cols; k += 64) {
    float gy = dyr[k] * bf16_to_f32(gain[k]);
    float a = r * gy;
    float b = xr[k] * q;
    dx[row * cols + k] = a - b;
  }
}

// dgain[k] = R1 over rows t of RN(dy[t,k] * RN(x[t,k] * rstd[t])).  A workgroup of 16 wavefronts takes 64
// columns (lane = column, so row reads are coalesced); wavefront q folds the aligned power-of-two group of
// row chunks [q*G, q*G + G), then the 16 group results are folded with the pass-through rule.
constexpr int kDgainGroups = 16;
__global__ __launch_bounds__(1024) void rownorm_dgain_kernel(int64_t rows, int64_t cols, const float* __restrict__ x,
                                                             const float* __restrict__ rstd,
                                                             const float* __restrict__ dy,
                                                             float* __restrict__ dgain) {
  __shared__ float part[kDgainGroups][64];
  const int lane = threadIdx.x & 63, grp = threadIdx.x >> 6;
  const int64_t col = (int64_t)blockIdx.x * 64 + lane;
  const int64_t nc = (rows + kChunk - 1) / kChunk;
  const int64_t G = block_chunks(nc, kDgainGroups);
  const int64_t c0 = grp * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  if (col < cols) {
    for (int64_t c = c0; c < c1; ++c) {
      float s = 0.0f;
      const int64_t t1 = (c + 1) * kChunk < rows ? (c + 1) * kChunk : rows;
      for (int64_t t = c * kChunk; t < t1; ++t) {
        float xh = x[t * cols + col] * rstd[t];
        float pr = dy[t * cols + col] * xh;
        s = s + pr;
      }
      f.push(s);
    }
  }
  part[grp][lane] = f.result();
  __syncthreads();
  if (grp == 0 && col < cols) {
    // fold the group results: level by level, a node adds its right neighbour when that subtree is real
    float v[kDgainGroups];
#pragma unroll
    for (int q = 0; q < kDgainGroups; ++q) v[q] = part[q][lane];
#pragma unroll
    for (int sdist = 1; sdist < kDgainGroups; sdist <<= 1)
#pragma unroll
      for (int q = 0; q + sdist < kDgainGroups; q += 2 * sdist)
        if ((q + sdist) * G < nc) v[q] = v[q] + v[q + sdist];
    dgain[col] = v[0];
  }
}

hipError_t rownorm_fwd_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, float eps, uint16_t* y,
                              float* rstd, hipStream_t s) {
  if (rows == 0) return hipSuccess;
  const float inv_d = (float)(1.0 / (double)cols);  // RN32(1/cols), correctly rounded
  hipLaunchKernelGGL(rownorm_fwd_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, rows, cols, x, gain, eps,
                     inv_d, y, rstd);
  return hipGetLastError();
}

hipError_t rownorm_bwd_launch(int64_t rows, int64_t cols, const float* x, const uint16_t* gain, const float* rstd,
                              const float* dy, float* dx, float* dgain, hipStream_t s) {
  if (rows == 0) {
    if (dgain) return hipMemsetAsync(dgain, 0, sizeof(float) * cols, s);
    return hipSuccess;
  }
  const float inv_d = (float)(1.0 / (double)cols);
  hipLaunchKernelGGL(rownorm_bwd_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, rows, cols, x, gain, rstd,
                     dy, inv_d, dx);
  if (dgain)
    hipLaunchKernelGGL(rownorm_dgain_kernel, dim3((unsigned)((cols + 63) / 64)), dim3(1024), 0, s, rows, cols, x,
                       rstd, dy, dgain);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// Causal softmax of raw scores: row r is query i = r mod cols; one wavefront per row, coalesced.
__global__ __launch_bounds__(256) void softmax_causal_kernel(int64_t rows, int64_t cols, const float* __restrict__ raw,
                                                             float scale, uint16_t* __restrict__ probs) {
  __shared__ WaveStage st[4];
  __shared__ float parts[4][kMaxRowChunks];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = (int64_t)blockIdx.x * 4 + w;
  if (row >= rows) return;
  const int64_t i = row % cols;
  const float* rr = raw + row * cols;
  float m = -__builtin_inff();
  for (int64_t j = lane; j <= i; j += 64) m = fmaxf(m, rr[j] * scale);
  m = wave_max(m);
  // masked keys enter the chain as +0 terms
  const float S = wave_row_rsum(cols, st[w], parts[w], [&](int64_t j) {
    float e = 0.0f;
    if (j <= i) {
      float sc = rr[j] * scale;
      e = cexp(sc - m);
    }
    return e;
  }, i + 1);
  const float rcp = 1.0f / S;
  for (int64_t j = lane; j < cols; j += 64) {
    uint16_t o = 0;
    if (j <= i) {
      float sc = rr[j] * scale;
      float e = cexp(sc - m);
      o = f32_to_bf16(e * rcp);
    }
    probs[row * cols + j] = o;
  }
}

hipError_t softmax_causal_launch(int64_t rows, int64_t cols, const float* raw, float scale, uint16_t* probs,
                                 hipStream_t s) {
  if (rows == 0) return hipSuccess;
  hipLaunchKernelGGL(softmax_causal_kernel, dim3((unsigned)((rows + 3) / 4)), dim3(256), 0, s, rows, cols, raw, scale,
                     probs);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// Cross-entropy: one 256-thread workgroup per row.  The four wavefronts take the row's 2048-term segments
// round-robin and write the chunk partials; the partials are then folded across the workgroup.
constexpr int kMaxXentChunks = 4096;  // vocabularies up to 131072
__global__ __launch_bounds__(256) void xent_kernel(int64_t rows, int64_t vocab, const uint16_t* __restrict__ logits,
                                                   const int32_t* __restrict__ targets, float inv_tokens,
                                                   uint16_t* __restrict__ dlogits, float* __restrict__ row_loss) {
  __shared__ WaveStage st[4];
  __shared__ float parts[kMaxXentChunks];
  __shared__ float red[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t row = blockIdx.x;
  const uint16_t* lr = logits + row * vocab;
  float m = -__builtin_inff();
  for (int64_t j = threadIdx.x; j < vocab; j += 256) m = fmaxf(m, bf16_to_f32(lr[j]));
  m = wave_max(m);
  if (lane == 0) red[w] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  for (int64_t seg0 = (int64_t)w * 64 * kChunk; seg0 < vocab; seg0 += 4 * 64 * kChunk)
    wave_segment_chunks(seg0, vocab, st[w], parts, [&](int64_t j) { return cexp(bf16_to_f32(lr[j]) - m); });
  __syncthreads();
  const int64_t nc = (vocab + kChunk - 1) / kChunk;
  const int64_t G = block_chunks(nc, 256);
  const int64_t c0 = threadIdx.x * G, c1 = (c0 + G < nc) ? c0 + G : nc;
  LocalFold f;
  for (int64_t c = c0; c < c1; ++c) f.push(parts[c]);
  const float S = block_fold(f.result(), (nc + G - 1) / G);
  const int32_t y = targets[row];
  const bool valid = y >= 0 && y < vocab;
  if (threadIdx.x == 0) {
    float lse = m + clog(S);
    row_loss[row] = valid ? lse - bf16_to_f32(lr[y]) : __builtin_nanf("");
  }
  const float rcp = 1.0f / S;
  if (dlogits) {
    for (int64_t j = threadIdx.x; j < vocab; j += 256) {
      float e = cexp(bf16_to_f32(lr[j]) - m);
      float p = e * rcp;
      float q = p - (j == y ? 1.0f : 0.0f);
      dlogits[row * vocab + j] = f32_to_bf16(q * inv_tokens);
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
                       uint16_t* dlogits, float* row_loss, float* mean_loss, hipStream_t s) {
  if (rows > 0)
    hipLaunchKernelGGL(xent_kernel, dim3((unsigned)rows), dim3(256), 0, s, rows, vocab, logits, targets, inv_tokens,
                       dlogits, row_loss);
  if (mean_loss)
    hipLaunchKernelGGL(mean_loss_kernel, dim3(1), dim3(256), 0, s, rows, row_loss, inv_tokens, mean_loss);
  return hipGetLastError();
}

// ------------------------------------------------------------------------------------------------
// D[bh][i] = R1 over d of fma(dO[i,d], O[i,d]) (bf16 operands, [T, ld] layout, head h at column h*hd).
__global__ __launch_bounds__(256) void attn_rowdot_kernel(int64_t B, int64_t H, int64_t S, int64_t hd,
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
    float s = 0.0f;
    const int64_t c1 = c0 + kChunk < hd ? c0 + kChunk : hd;
    for (int64_t k = c0; k < c1; ++k) s = __builtin_fmaf(bf16_to_f32(a[k]), bf16_to_f32(o[k]), s);
    f.push(s);
  }
  D[idx] = f.result();
}

hipError_t attn_rowdot_launch(int64_t B, int64_t H, int64_t S, int64_t hd, const uint16_t* dO, const uint16_t* O,
                              int64_t ld, float* D, hipStream_t s) {
  const int64_t n = B * H * S;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_rowdot_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, B, H, S, hd, dO, O, ld,
                     D);
  return hipGetLastError();
}

// dS = bf16(RN(RN(P * RN(dP - D)) * scale)) for j <= i, +0 for masked keys.
__global__ __launch_bounds__(256) void attn_dS_kernel(int64_t BH, int64_t S, const uint16_t* __restrict__ P,
                                                      const float* __restrict__ dP, const float* __restrict__ D,
                                                      float scale, uint16_t* __restrict__ dS) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t total = BH * S * S;
  if (idx >= total) return;
  const int64_t j = idx % S, row = idx / S, i = row % S;
  uint16_t o = 0;
  if (j <= i) {
    float t = dP[idx] - D[row];
    float u = bf16_to_f32(P[idx]) * t;
    o = f32_to_bf16(u * scale);
  }
  dS[idx] = o;
}

hipError_t attn_dS_launch(int64_t BH, int64_t S, const uint16_t* P, const float* dP, const float* D, float scale,
                          uint16_t* dS, hipStream_t s) {
  const int64_t n = BH * S * S;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(attn_dS_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, BH, S, P, dP, D, scale, dS);
  return hipGetLastError();
}

}  // namespace canon
