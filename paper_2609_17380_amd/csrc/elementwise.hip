// elementwise.hip - RoPE (R8), SwiGLU (R4), residual adds and casts (R10), embedding gather and the
// ordered embedding backward (R11), and a device-math probe for the primitives.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

static inline unsigned blocks_for(int64_t n) { return (unsigned)((n + 255) / 256); }

// The fused projection qkv [T][N], N = (H + 2 Hkv) hd, holds H query heads, then Hkv key heads, then Hkv
// value heads.  Head slot u < H + Hkv names query head u (u < H) or key head u - H; both are rotated at
// their position and stored bf16 head-major (q [B][H][S][hd], k and v [B][Hkv][S][hd]); the key slots also
// copy their value head.
__global__ void rope_qkv_kernel(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd,
                                const float* __restrict__ qkv, const float* __restrict__ cosT,
                                const float* __restrict__ sinT, uint16_t* __restrict__ q, uint16_t* __restrict__ k,
                                uint16_t* __restrict__ v) {
  const int64_t hh = hd / 2, U = H + Hkv, N = (H + 2 * Hkv) * hd;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S * U * hh) return;
  const int64_t i = idx % hh, u = (idx / hh) % U, t = idx / (hh * U);
  const int64_t b = t / S, s = t % S;
  const float c = cosT[s * hh + i], sn = sinT[s * hh + i];
  const float* row = qkv + t * N + u * hd;
  uint16_t* out = u < H ? q + ((b * H + u) * S + s) * hd : k + ((b * Hkv + (u - H)) * S + s) * hd;
  float x1 = row[i], x2 = row[i + hh];
  float a = x1 * c, bq = x2 * sn;
  float e = x2 * c, f = x1 * sn;
  out[i] = f32_to_bf16(a - bq);
  out[i + hh] = f32_to_bf16(e + f);
  if (u >= H) {
    const float* vr = row + Hkv * hd;
    uint16_t* vo = v + ((b * Hkv + (u - H)) * S + s) * hd;
    vo[i] = f32_to_bf16(vr[i]);
    vo[i + hh] = f32_to_bf16(vr[i + hh]);
  }
}

// The same with the gain-free QK-norm before the rotation: one thread per head row.  r = 1 / sqrt(RN(ms +
// eps)) with ms = RN(R1(x^2) * RN(1/hd)) (chains of 32, Algorithm 2), saved per row in rq [T][H + Hkv];
// the normalised row RN(x * r) stays fp32 into the rotation.
__global__ void rope_qkv_norm_kernel(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd,
                                     const float* __restrict__ qkv, const float* __restrict__ cosT,
                                     const float* __restrict__ sinT, float eps, float inv_hd,
                                     uint16_t* __restrict__ q, uint16_t* __restrict__ k, uint16_t* __restrict__ v,
                                     float* __restrict__ rq) {
  const int64_t hh = hd / 2, U = H + Hkv, N = (H + 2 * Hkv) * hd;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S * U) return;
  const int64_t u = idx % U, t = idx / U;
  const int64_t b = t / S, s = t % S;
  const float* row = qkv + t * N + u * hd;
  LocalFoldN<8> fold;
  for (int64_t c0 = 0; c0 < hd; c0 += kChunk) {
    const int64_t c1 = c0 + kChunk < hd ? c0 + kChunk : hd;
    float acc = 0.0f;
    for (int64_t j = c0; j < c1; ++j) {
      const float xj = row[j];
      acc = acc + xj * xj;
    }
    fold.push(acc);
  }
  const float ms = fold.result() * inv_hd;
  const float var = ms + eps;
  const float r = 1.0f / __builtin_sqrtf(var);
  rq[idx] = r;
  uint16_t* out = u < H ? q + ((b * H + u) * S + s) * hd : k + ((b * Hkv + (u - H)) * S + s) * hd;
  for (int64_t i = 0; i < hh; ++i) {
    const float c = cosT[s * hh + i], sn = sinT[s * hh + i];
    const float x1 = row[i] * r, x2 = row[i + hh] * r;
    float a = x1 * c, bq = x2 * sn;
    float e = x2 * c, f = x1 * sn;
    out[i] = f32_to_bf16(a - bq);
    out[i + hh] = f32_to_bf16(e + f);
  }
  if (u >= H) {
    const float* vr = row + Hkv * hd;
    uint16_t* vo = v + ((b * Hkv + (u - H)) * S + s) * hd;
    for (int64_t j = 0; j < hd; ++j) vo[j] = f32_to_bf16(vr[j]);
  }
}

// Wavefront-per-segment QK-norm (head size HD = 64, 128 or 256).  A segment is up to 2048 consecutive floats
// of one token's q part (H heads) or k part (Hkv heads): whole heads, read coalesced, lane l holding
// elements 256 q + 4 l .. +3.  Squares (or, backward, the products gy * x) are staged transposed in LDS so
// that lane c runs chunk c's chain; the HD / 32 chunks of a head fold by shuffles (a complete subtree), and
// the rotation's partner element i +- HD/2 sits in lane l ^ (HD / 8).
struct QkStage {
  float t[64][33];
};

__device__ __forceinline__ void qk_item(int64_t item, int64_t nsq, int64_t nsk, int64_t& t, int& part, int64_t& seg) {
  const int64_t per = nsq + nsk;
  t = item / per;
  const int64_t r = item % per;
  part = r < nsq ? 0 : 1;
  seg = part == 0 ? r : r - nsq;
}

// chains of the staged segment (len floats) and the per-head fold: lane h * (HD / 32) returns head h's sum
template <int HD>
__device__ __forceinline__ float qk_head_sums(QkStage& st, int64_t len) {
  constexpr int CPH = HD / 32;
  const int lane = threadIdx.x & 63;
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  float p = 0.0f;
  if (lane < len / kChunk) {
    for (int i = 0; i < kChunk; ++i) p = p + st.t[lane][i];
  }
#pragma unroll
  for (int sft = 1; sft < CPH; sft <<= 1) {
    const float o = __shfl_down(p, sft, 64);
    if ((lane & (2 * sft - 1)) == 0) p = p + o;
  }
  __builtin_amdgcn_s_waitcnt(0);
  __builtin_amdgcn_wave_barrier();
  return p;
}

template <int HD>
__global__ __launch_bounds__(256) void rope_qkv_norm_wave_kernel(int64_t B, int64_t S, int64_t H, int64_t Hkv,
                                                                 const float* __restrict__ qkv,
                                                                 const float* __restrict__ cosT,
                                                                 const float* __restrict__ sinT, float eps,
                                                                 float inv_hd, uint16_t* __restrict__ q,
                                                                 uint16_t* __restrict__ k, uint16_t* __restrict__ v,
                                                                 float* __restrict__ rq) {
  constexpr int CPH = HD / 32, HH = HD / 2;
  __shared__ QkStage stage[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t N = (H + 2 * Hkv) * HD;
  const int64_t nsq = (H * HD + 2047) / 2048, nsk = (Hkv * HD + 2047) / 2048;
  const int64_t item = (int64_t)blockIdx.x * 4 + w;
  if (item >= B * S * (nsq + nsk)) return;
  int64_t t, seg;
  int part;
  qk_item(item, nsq, nsk, t, part, seg);
  const int64_t b = t / S, s = t % S;
  const int64_t nh = part == 0 ? H : Hkv;
  const int64_t len = (nh * HD - seg * 2048) < 2048 ? nh * HD - seg * 2048 : 2048;
  const int64_t head0 = seg * (2048 / HD);
  const float* src = qkv + t * N + (part == 0 ? 0 : H * HD) + seg * 2048;
  float x[8][4];
#pragma unroll
  for (int qq = 0; qq < 8; ++qq) {
    const int64_t e = 256 * qq + 4 * lane;
    float4 f4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if (e < len) f4 = *reinterpret_cast<const float4*>(src + e);
    x[qq][0] = f4.x; x[qq][1] = f4.y; x[qq][2] = f4.z; x[qq][3] = f4.w;
    if (e < len) {
      float* dst = &stage[w].t[e >> 5][e & 31];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) dst[kk] = x[qq][kk] * x[qq][kk];
    }
  }
  const float ss = qk_head_sums<HD>(stage[w], len);
  float r = 0.0f;
  if ((lane % CPH) == 0 && lane < len / kChunk) {
    const float ms = ss * inv_hd;
    const float var = ms + eps;
    r = 1.0f / __builtin_sqrtf(var);
    rq[t * (H + Hkv) + (part == 0 ? 0 : H) + head0 + lane / CPH] = r;
  }
  uint16_t* outb = part == 0 ? q : k;
#pragma unroll
  for (int qq = 0; qq < 8; ++qq) {
    const int64_t e = 256 * qq + 4 * lane;
    const int hl = (int)((256 * qq + 4 * lane) / HD);
    const float rr = __shfl(r, (hl * CPH) & 63, 64);
    float xn[4], xp[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) xn[kk] = x[qq][kk] * rr;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) xp[kk] = __shfl_xor(xn[kk], HD / 8, 64);
    if (e < len) {
      const int i0 = (int)((256 * qq + 4 * lane) % HD);
      uint16_t o[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const int i = i0 + kk, ih = i % HH;
        const float c = cosT[s * HH + ih], sn = sinT[s * HH + ih];
        const float a = xn[kk] * c, bb = xp[kk] * sn;
        o[kk] = f32_to_bf16(i < HH ? a - bb : a + bb);
      }
      uint16_t* dst = outb + ((b * nh + head0 + hl) * S + s) * HD + i0;
      *reinterpret_cast<uint2*>(dst) = make_uint2((uint32_t)o[0] | ((uint32_t)o[1] << 16),
                                                  (uint32_t)o[2] | ((uint32_t)o[3] << 16));
    }
  }
  if (part == 1) {  // the value heads of this segment
    const float* vs = qkv + t * N + (H + Hkv) * HD + seg * 2048;
#pragma unroll
    for (int qq = 0; qq < 8; ++qq) {
      const int64_t e = 256 * qq + 4 * lane;
      if (e < len) {
        const float4 f4 = *reinterpret_cast<const float4*>(vs + e);
        const int hl = (int)(e / HD), i0 = (int)(e % HD);
        uint16_t* dst = v + ((b * Hkv + head0 + hl) * S + s) * HD + i0;
        *reinterpret_cast<uint2*>(dst) =
            make_uint2((uint32_t)f32_to_bf16(f4.x) | ((uint32_t)f32_to_bf16(f4.y) << 16),
                       (uint32_t)f32_to_bf16(f4.z) | ((uint32_t)f32_to_bf16(f4.w) << 16));
      }
    }
  }
}

template <int HD>
__global__ __launch_bounds__(256) void rope_bwd_norm_wave_kernel(int64_t B, int64_t S, int64_t H, int64_t Hkv,
                                                                 const float* __restrict__ dq,
                                                                 const float* __restrict__ dk,
                                                                 const float* __restrict__ qkv,
                                                                 const float* __restrict__ rq,
                                                                 const float* __restrict__ cosT,
                                                                 const float* __restrict__ sinT, float inv_hd,
                                                                 uint16_t* __restrict__ dqkv) {
  constexpr int CPH = HD / 32, HH = HD / 2;
  __shared__ QkStage stage[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t N = (H + 2 * Hkv) * HD;
  const int64_t nsq = (H * HD + 2047) / 2048, nsk = (Hkv * HD + 2047) / 2048;
  const int64_t item = (int64_t)blockIdx.x * 4 + w;
  if (item >= B * S * (nsq + nsk)) return;
  int64_t t, seg;
  int part;
  qk_item(item, nsq, nsk, t, part, seg);
  const int64_t s = t % S;
  const int64_t nh = part == 0 ? H : Hkv;
  const int64_t len = (nh * HD - seg * 2048) < 2048 ? nh * HD - seg * 2048 : 2048;
  const int64_t head0 = seg * (2048 / HD);
  const float* gsrc = part == 0 ? dq + t * H * HD + seg * 2048 : dk + t * Hkv * HD + seg * 2048;
  const int64_t col0 = (part == 0 ? 0 : H * HD) + seg * 2048;
  const float* xsrc = qkv + t * N + col0;
  float gy[8][4], x[8][4];
#pragma unroll
  for (int qq = 0; qq < 8; ++qq) {
    const int64_t e = 256 * qq + 4 * lane;
    float4 g4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f), x4 = g4;
    if (e < len) {
      g4 = *reinterpret_cast<const float4*>(gsrc + e);
      x4 = *reinterpret_cast<const float4*>(xsrc + e);
    }
    const float g[4] = {g4.x, g4.y, g4.z, g4.w};
    x[qq][0] = x4.x; x[qq][1] = x4.y; x[qq][2] = x4.z; x[qq][3] = x4.w;
    float gp[4];
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) gp[kk] = __shfl_xor(g[kk], HD / 8, 64);
    const int i0 = (int)((256 * qq + 4 * lane) % HD);
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int i = i0 + kk, ih = i % HH;
      const float c = (e < len) ? cosT[s * HH + ih] : 0.0f, sn = (e < len) ? sinT[s * HH + ih] : 0.0f;
      const float a = g[kk] * c, bb = gp[kk] * sn;
      gy[qq][kk] = i < HH ? a + bb : a - bb;
    }
    if (e < len) {
      float* dst = &stage[w].t[e >> 5][e & 31];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) dst[kk] = gy[qq][kk] * x[qq][kk];
    }
  }
  const float dot = qk_head_sums<HD>(stage[w], len);
  float r = 0.0f, qc = 0.0f;
  if ((lane % CPH) == 0 && lane < len / kChunk) {
    r = rq[t * (H + Hkv) + (part == 0 ? 0 : H) + head0 + lane / CPH];
    const float r2 = r * r;
    const float r3 = r2 * r;
    const float dm = dot * inv_hd;
    qc = r3 * dm;
  }
#pragma unroll
  for (int qq = 0; qq < 8; ++qq) {
    const int64_t e = 256 * qq + 4 * lane;
    const int hl = (int)((256 * qq + 4 * lane) / HD);
    const float rr = __shfl(r, (hl * CPH) & 63, 64);
    const float qh = __shfl(qc, (hl * CPH) & 63, 64);
    if (e < len) {
      uint16_t o[4];
#pragma unroll
      for (int kk = 0; kk < 4; ++kk) {
        const float a = rr * gy[qq][kk], bb = x[qq][kk] * qh;
        o[kk] = f32_to_bf16(a - bb);
      }
      uint16_t* dst = dqkv + t * N + col0 + e;
      *reinterpret_cast<uint2*>(dst) = make_uint2((uint32_t)o[0] | ((uint32_t)o[1] << 16),
                                                  (uint32_t)o[2] | ((uint32_t)o[3] << 16));
    }
  }
}

static bool qk_wave_ok(int64_t H, int64_t Hkv, int64_t hd, const void* a, const void* b) {
  return (hd == 64 || hd == 128 || hd == 256) && ((uintptr_t)a & 15) == 0 && ((uintptr_t)b & 7) == 0 && H > 0 &&
         Hkv > 0;
}

hipError_t rope_qkv_launch(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd, const float* qkv,
                           const float* cosT, const float* sinT, int qk_norm, float eps, uint16_t* q, uint16_t* k,
                           uint16_t* v, float* rq, hipStream_t s) {
  if (qk_norm) {
    const int64_t n = B * S * (H + Hkv);
    if (n == 0) return hipSuccess;
    const float inv_hd = (float)(1.0 / (double)hd);  // RN32(1/hd)
    if (qk_wave_ok(H, Hkv, hd, qkv, q) && ((uintptr_t)k & 7) == 0 && ((uintptr_t)v & 7) == 0) {
      const int64_t items = B * S * ((H * hd + 2047) / 2048 + (Hkv * hd + 2047) / 2048);
      const dim3 grid((unsigned)((items + 3) / 4));
      if (hd == 64)
        hipLaunchKernelGGL(rope_qkv_norm_wave_kernel<64>, grid, dim3(256), 0, s, B, S, H, Hkv, qkv, cosT, sinT, eps,
                           inv_hd, q, k, v, rq);
      else if (hd == 128)
        hipLaunchKernelGGL(rope_qkv_norm_wave_kernel<128>, grid, dim3(256), 0, s, B, S, H, Hkv, qkv, cosT, sinT, eps,
                           inv_hd, q, k, v, rq);
      else
        hipLaunchKernelGGL(rope_qkv_norm_wave_kernel<256>, grid, dim3(256), 0, s, B, S, H, Hkv, qkv, cosT, sinT, eps,
                           inv_hd, q, k, v, rq);
      return hipGetLastError();
    }
    hipLaunchKernelGGL(rope_qkv_norm_kernel, dim3(blocks_for(n)), dim3(256), 0, s, B, S, H, Hkv, hd, qkv, cosT, sinT,
                       eps, inv_hd, q, k, v, rq);
    return hipGetLastError();
  }
  const int64_t n = B * S * (H + Hkv) * (hd / 2);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_qkv_kernel, dim3(blocks_for(n)), dim3(256), 0, s, B, S, H, Hkv, hd, qkv, cosT, sinT, q, k,
                     v);
  return hipGetLastError();
}

// Transposed rotation of the q and k gradients (dq [T][H hd], dk [T][Hkv hd], fp32) into the q and k columns
// of dqkv (bf16 [T][N]).
__global__ void rope_bwd_kernel(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd,
                                const float* __restrict__ dq, const float* __restrict__ dk,
                                const float* __restrict__ cosT, const float* __restrict__ sinT,
                                uint16_t* __restrict__ dqkv) {
  const int64_t hh = hd / 2, U = H + Hkv, N = (H + 2 * Hkv) * hd;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S * U * hh) return;
  const int64_t i = idx % hh, u = (idx / hh) % U, t = idx / (hh * U);
  const int64_t s = t % S;
  const float c = cosT[s * hh + i], sn = sinT[s * hh + i];
  const float* g = u < H ? dq + t * H * hd + u * hd : dk + t * Hkv * hd + (u - H) * hd;
  float g1 = g[i], g2 = g[i + hh];
  float a = g1 * c, b = g2 * sn;
  float e = g2 * c, f = g1 * sn;
  dqkv[t * N + u * hd + i] = f32_to_bf16(a + b);
  dqkv[t * N + u * hd + i + hh] = f32_to_bf16(e - f);
}

// element j of the transposed rotation of head row g at position s
__device__ __forceinline__ float rope_bwd_elem(const float* g, const float* cs, const float* sn, int64_t hh,
                                               int64_t j) {
  if (j < hh) {
    const float a = g[j] * cs[j], b = g[j + hh] * sn[j];
    return a + b;
  }
  const int64_t i = j - hh;
  const float e = g[j] * cs[i], f = g[i] * sn[i];
  return e - f;
}

// With QK-norm: the transposed rotation, then R3's input gradient without a gain (dot = R1(gy * x), q =
// RN(RN(RN(r r) r) RN(dot / hd)), dx = RN(RN(r gy) - RN(x q))), one thread per head row.
__global__ void rope_bwd_norm_kernel(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd,
                                     const float* __restrict__ dq, const float* __restrict__ dk,
                                     const float* __restrict__ qkv, const float* __restrict__ rq,
                                     const float* __restrict__ cosT, const float* __restrict__ sinT, float inv_hd,
                                     uint16_t* __restrict__ dqkv) {
  const int64_t hh = hd / 2, U = H + Hkv, N = (H + 2 * Hkv) * hd;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S * U) return;
  const int64_t u = idx % U, t = idx / U, s = t % S;
  const float* g = u < H ? dq + t * H * hd + u * hd : dk + t * Hkv * hd + (u - H) * hd;
  const float* x = qkv + t * N + u * hd;
  const float* cs = cosT + s * hh;
  const float* sn = sinT + s * hh;
  const float r = rq[idx];
  LocalFoldN<8> fold;
  for (int64_t c0 = 0; c0 < hd; c0 += kChunk) {
    const int64_t c1 = c0 + kChunk < hd ? c0 + kChunk : hd;
    float acc = 0.0f;
    for (int64_t j = c0; j < c1; ++j) {
      const float p = rope_bwd_elem(g, cs, sn, hh, j) * x[j];
      acc = acc + p;
    }
    fold.push(acc);
  }
  const float dot = fold.result();
  const float r2 = r * r;
  const float r3 = r2 * r;
  const float dm = dot * inv_hd;
  const float qc = r3 * dm;
  for (int64_t j = 0; j < hd; ++j) {
    const float gy = rope_bwd_elem(g, cs, sn, hh, j);
    const float a = r * gy, b = x[j] * qc;
    dqkv[t * N + u * hd + j] = f32_to_bf16(a - b);
  }
}

hipError_t rope_bwd_launch(int64_t B, int64_t S, int64_t H, int64_t Hkv, int64_t hd, const float* dq, const float* dk,
                           const float* cosT, const float* sinT, int qk_norm, const float* qkv, const float* rq,
                           uint16_t* dqkv, hipStream_t s) {
  if (qk_norm) {
    const int64_t n = B * S * (H + Hkv);
    if (n == 0) return hipSuccess;
    const float inv_hd = (float)(1.0 / (double)hd);
    if (qk_wave_ok(H, Hkv, hd, qkv, dqkv) && ((uintptr_t)dq & 15) == 0 && ((uintptr_t)dk & 15) == 0) {
      const int64_t items = B * S * ((H * hd + 2047) / 2048 + (Hkv * hd + 2047) / 2048);
      const dim3 grid((unsigned)((items + 3) / 4));
      if (hd == 64)
        hipLaunchKernelGGL(rope_bwd_norm_wave_kernel<64>, grid, dim3(256), 0, s, B, S, H, Hkv, dq, dk, qkv, rq, cosT,
                           sinT, inv_hd, dqkv);
      else if (hd == 128)
        hipLaunchKernelGGL(rope_bwd_norm_wave_kernel<128>, grid, dim3(256), 0, s, B, S, H, Hkv, dq, dk, qkv, rq, cosT,
                           sinT, inv_hd, dqkv);
      else
        hipLaunchKernelGGL(rope_bwd_norm_wave_kernel<256>, grid, dim3(256), 0, s, B, S, H, Hkv, dq, dk, qkv, rq, cosT,
                           sinT, inv_hd, dqkv);
      return hipGetLastError();
    }
    hipLaunchKernelGGL(rope_bwd_norm_kernel, dim3(blocks_for(n)), dim3(256), 0, s, B, S, H, Hkv, hd, dq, dk, qkv, rq,
                       cosT, sinT, inv_hd, dqkv);
    return hipGetLastError();
  }
  const int64_t n = B * S * (H + Hkv) * (hd / 2);
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(rope_bwd_kernel, dim3(blocks_for(n)), dim3(256), 0, s, B, S, H, Hkv, hd, dq, dk, cosT, sinT,
                     dqkv);
  return hipGetLastError();
}

// dO [T][H hd] (token-major) -> head-major [B][H][S][hd], bf16: the grouped heads' value gradient reads a
// group's dO as one stacked operand
__global__ void heads_major_kernel(int64_t B, int64_t S, int64_t H, int64_t hd, const uint16_t* __restrict__ src,
                                   uint16_t* __restrict__ dst) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S * H * hd) return;
  const int64_t j = idx % hd, h = (idx / hd) % H, t = idx / (hd * H);
  const int64_t b = t / S, s = t % S;
  dst[((b * H + h) * S + s) * hd + j] = src[idx];
}

hipError_t heads_major_launch(int64_t B, int64_t S, int64_t H, int64_t hd, const uint16_t* src, uint16_t* dst,
                              hipStream_t s) {
  const int64_t n = B * S * H * hd;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(heads_major_kernel, dim3(blocks_for(n)), dim3(256), 0, s, B, S, H, hd, src, dst);
  return hipGetLastError();
}

// a = bf16(RN(silu(gate) * up)); gu = [T, 2F] with gate columns first.
__global__ void swiglu_fwd_kernel(int64_t T, int64_t F, const float* __restrict__ gu, uint16_t* __restrict__ a) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= T * F) return;
  const int64_t t = idx / F, j = idx % F;
  float g = gu[t * 2 * F + j], u = gu[t * 2 * F + F + j];
  float sl = csilu(g);
  a[idx] = f32_to_bf16(sl * u);
}

__global__ void swiglu_bwd_kernel(int64_t T, int64_t F, const float* __restrict__ gu, const float* __restrict__ da,
                                  uint16_t* __restrict__ dgu) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= T * F) return;
  const int64_t t = idx / F, j = idx % F;
  float g = gu[t * 2 * F + j], u = gu[t * 2 * F + F + j], dav = da[idx];
  float sig = csigmoid(g);
  float sl = g * sig;
  float dup = dav * sl;
  float oms = 1.0f - sig;
  float gs = g * oms;
  float ops = 1.0f + gs;
  float dsg = sig * ops;
  float du = dav * u;
  float dgate = du * dsg;
  dgu[t * 2 * F + j] = f32_to_bf16(dgate);
  dgu[t * 2 * F + F + j] = f32_to_bf16(dup);
}

hipError_t swiglu_fwd_launch(int64_t T, int64_t F, const float* gu, uint16_t* a, hipStream_t s) {
  if (T * F == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_fwd_kernel, dim3(blocks_for(T * F)), dim3(256), 0, s, T, F, gu, a);
  return hipGetLastError();
}

hipError_t swiglu_bwd_launch(int64_t T, int64_t F, const float* gu, const float* da, uint16_t* dgu, hipStream_t s) {
  if (T * F == 0) return hipSuccess;
  hipLaunchKernelGGL(swiglu_bwd_kernel, dim3(blocks_for(T * F)), dim3(256), 0, s, T, F, gu, da, dgu);
  return hipGetLastError();
}

__global__ void add_f32_kernel(int64_t n, const float* __restrict__ a, const float* __restrict__ b, float* out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) out[i] = a[i] + b[i];
}

__global__ void cast_bf16_kernel(int64_t n, const float* __restrict__ x, uint16_t* __restrict__ y) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = f32_to_bf16(x[i]);
}

__global__ void widen_bf16_kernel(int64_t n, const uint16_t* __restrict__ x, float* __restrict__ y) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) y[i] = bf16_to_f32(x[i]);
}

hipError_t add_f32_launch(int64_t n, const float* a, const float* b, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(add_f32_kernel, dim3(blocks_for(n)), dim3(256), 0, s, n, a, b, out);
  return hipGetLastError();
}

hipError_t cast_bf16_launch(int64_t n, const float* x, uint16_t* y, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(cast_bf16_kernel, dim3(blocks_for(n)), dim3(256), 0, s, n, x, y);
  return hipGetLastError();
}

hipError_t widen_bf16_launch(int64_t n, const uint16_t* x, float* y, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(widen_bf16_kernel, dim3(blocks_for(n)), dim3(256), 0, s, n, x, y);
  return hipGetLastError();
}

__global__ void token_check_kernel(int64_t n, const int32_t* __restrict__ tok, int32_t bound, int32_t* flag) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n && (tok[i] < 0 || tok[i] >= bound)) atomicOr(flag, 1);
}

hipError_t token_check_launch(int64_t n, const int32_t* tok, int32_t bound, int32_t* flag, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(token_check_kernel, dim3(blocks_for(n)), dim3(256), 0, s, n, tok, bound, flag);
  return hipGetLastError();
}

// x[b*S + s, :] = widen(E[win[b, s], :]); an out-of-range token gives a zero row (the step reports it).
__global__ void embed_gather_kernel(int64_t B, int64_t S, int64_t d, const int32_t* __restrict__ win, int64_t win_ld,
                                    const uint16_t* __restrict__ E, int64_t V, float* __restrict__ x) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S * d) return;
  const int64_t k = idx % d, t = idx / d, b = t / S, s = t % S;
  const int32_t tok = win[b * win_ld + s];
  x[idx] = (tok >= 0 && tok < V) ? bf16_to_f32(E[(int64_t)tok * d + k]) : 0.0f;
}

hipError_t embed_gather_launch(int64_t B, int64_t S, int64_t d, const int32_t* win, int64_t win_ld, const uint16_t* E,
                               int64_t V, float* x, hipStream_t s) {
  const int64_t n = B * S * d;
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(embed_gather_kernel, dim3(blocks_for(n)), dim3(256), 0, s, B, S, d, win, win_ld, E, V, x);
  return hipGetLastError();
}

__global__ void labels_kernel(int64_t B, int64_t S, const int32_t* __restrict__ win, int64_t win_ld,
                              int32_t* __restrict__ lab) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= B * S) return;
  const int64_t b = idx / S, s = idx % S;
  lab[idx] = win[b * win_ld + s + 1];
}

hipError_t labels_launch(int64_t B, int64_t S, const int32_t* win, int64_t win_ld, int32_t* lab, hipStream_t s) {
  if (B * S == 0) return hipSuccess;
  hipLaunchKernelGGL(labels_kernel, dim3(blocks_for(B * S)), dim3(256), 0, s, B, S, win, win_ld, lab);
  return hipGetLastError();
}

// ---- embedding backward (R11) ----------------------------------------------------------------------
// dE[v] = R1 over the ascending positions t with tok[t] = v of dx[t].
//  1. Keys key[t] = (uint32 token) << 32 | t, padded with ~0 to a power of two.  Every key is distinct, so
//     the sorted order is unique: tokens ascending, positions ascending within a token (no atomics, no
//     tie order to fix).
//  2. Bitonic sort of the keys: blocks of kSortBlk keys sorted in LDS, then for each larger merge size the
//     steps with a partner distance of kSortBlk or more in global memory and the rest in LDS.
//  3. Segment starts: one workgroup max-scans the head flags of the sorted slots.
//  4. Chunk chains: one workgroup per sorted slot that starts a chunk (its distance from the segment start
//     a multiple of 32) runs the chain of its <= 32 positions for every column; a segment of one chunk writes
//     dE directly, longer segments write the chain partial to part[slot].
//  5. Fold: one workgroup per segment of more than one chunk folds its chunk partials by Algorithm 2.
// Tokens outside [0, V) sort after every valid token and contribute nothing.
constexpr int kSortBlk = 2048;  // keys per LDS sort block (16 KB), one compare-exchange per thread per step

__device__ __forceinline__ int32_t tok_at(const int32_t* win, int64_t win_ld, int64_t S, int64_t t) {
  return win[(t / S) * win_ld + (t % S)];
}

static int64_t sort_len(int64_t T) {
  int64_t P = 2;
  while (P < T) P <<= 1;
  return P;
}

__global__ void embed_keys_kernel(int64_t T, int64_t P, int64_t S, const int32_t* __restrict__ win, int64_t win_ld,
                                  uint64_t* __restrict__ keys) {
  const int64_t t = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t >= P) return;
  keys[t] = t < T ? ((uint64_t)(uint32_t)tok_at(win, win_ld, S, t) << 32) | (uint64_t)t : ~uint64_t(0);
}

// one compare-exchange of the bitonic network at merge size k, partner distance j, for pair q
__device__ __forceinline__ void bitonic_pair(uint64_t* a, int64_t base, int64_t q, int64_t k, int64_t j) {
  const int64_t i = 2 * j * (q / j) + (q % j), l = i + j;
  const bool up = ((base + i) & k) == 0;
  const uint64_t x = a[i], y = a[l];
  if (up ? (x > y) : (x < y)) {
    a[i] = y;
    a[l] = x;
  }
}

// blk = min(P, kSortBlk) keys per workgroup.  k == 0: sort each block completely (merge sizes 2 .. blk);
// otherwise the steps j = blk/2 .. 1 of merge size k.
__global__ __launch_bounds__(1024) void bitonic_local_kernel(uint64_t* __restrict__ keys, int64_t blk, int64_t k) {
  __shared__ uint64_t a[kSortBlk];
  const int64_t base = (int64_t)blockIdx.x * blk;
  for (int64_t i = threadIdx.x; i < blk; i += 1024) a[i] = keys[base + i];
  __syncthreads();
  const int64_t k0 = k == 0 ? 2 : k, k1 = k == 0 ? blk : k;
  for (int64_t kk = k0; kk <= k1; kk <<= 1) {
    for (int64_t j = (k == 0 ? kk : blk) >> 1; j > 0; j >>= 1) {
      for (int64_t q = threadIdx.x; q < blk / 2; q += 1024) bitonic_pair(a, base, q, kk, j);
      __syncthreads();
    }
  }
  for (int64_t i = threadIdx.x; i < blk; i += 1024) keys[base + i] = a[i];
}

__global__ void bitonic_global_kernel(uint64_t* __restrict__ keys, int64_t P, int64_t k, int64_t j) {
  const int64_t q = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (q >= P / 2) return;
  bitonic_pair(keys, 0, q, k, j);
}

// seg[p] = the first sorted slot of p's token, for p < T (one workgroup of 1024 threads)
__global__ __launch_bounds__(1024) void embed_segstart_kernel(int64_t T, const uint64_t* __restrict__ keys,
                                                              int32_t* __restrict__ seg) {
  __shared__ int64_t pre[1024];
  const int64_t per = (T + 1023) / 1024, p0 = (int64_t)threadIdx.x * per;
  int64_t run = 0;
  for (int64_t p = p0; p < p0 + per && p < T; ++p)
    if (p == 0 || (keys[p] >> 32) != (keys[p - 1] >> 32)) run = p;
  pre[threadIdx.x] = run;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {  // inclusive max-scan of the thread maxima
    const int64_t o = threadIdx.x >= (unsigned)off ? pre[threadIdx.x - off] : 0;
    __syncthreads();
    if (o > pre[threadIdx.x]) pre[threadIdx.x] = o;
    __syncthreads();
  }
  run = threadIdx.x > 0 ? pre[threadIdx.x - 1] : 0;
  for (int64_t p = p0; p < p0 + per && p < T; ++p) {
    if (p == 0 || (keys[p] >> 32) != (keys[p - 1] >> 32)) run = p;
    seg[p] = (int32_t)run;
  }
}

// VEC: four columns per thread with 16-byte loads (d % 4 == 0, dx, dE and part 16-byte aligned)
template <bool VEC>
__global__ __launch_bounds__(256) void embed_chunk_kernel(int64_t T, int64_t d, int64_t V,
                                                          const uint64_t* __restrict__ keys,
                                                          const int32_t* __restrict__ seg,
                                                          const float* __restrict__ dx, float* __restrict__ dE,
                                                          float* __restrict__ part) {
  const int64_t p = blockIdx.x;
  const int64_t ss = seg[p];
  if ((p - ss) % kChunk != 0) return;  // not the first slot of a chunk
  const uint64_t v = keys[p] >> 32;
  if (v >= (uint64_t)V) return;
  __shared__ int32_t pos[kChunk];
  if (threadIdx.x < kChunk) {
    const int64_t q = p + threadIdx.x;
    pos[threadIdx.x] = (q < T && (keys[q] >> 32) == v) ? (int32_t)(uint32_t)keys[q] : -1;
  }
  __syncthreads();
  int len = 0;
  while (len < kChunk && pos[len] >= 0) ++len;
  const bool more = p + kChunk < T && (keys[p + kChunk] >> 32) == v;
  float* out = (p == ss && !more) ? dE + (int64_t)v * d : part + p * d;  // one chunk: the result itself
  if (VEC) {
    for (int64_t k = 4 * (int64_t)threadIdx.x; k < d; k += 1024) {
      float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      for (int i = 0; i < len; ++i) {
        const float4 g = *reinterpret_cast<const float4*>(dx + (int64_t)pos[i] * d + k);
        acc.x = acc.x + g.x;
        acc.y = acc.y + g.y;
        acc.z = acc.z + g.z;
        acc.w = acc.w + g.w;
      }
      *reinterpret_cast<float4*>(out + k) = acc;
    }
  } else {
    for (int64_t k = threadIdx.x; k < d; k += 256) {
      float acc = 0.0f;
      for (int i = 0; i < len; ++i) acc = acc + dx[(int64_t)pos[i] * d + k];
      out[k] = acc;
    }
  }
}

// one workgroup per segment of more than one chunk: Algorithm 2 over its chunk partials, per column
__global__ __launch_bounds__(256) void embed_fold_kernel(int64_t T, int64_t d, int64_t V,
                                                         const uint64_t* __restrict__ keys,
                                                         const int32_t* __restrict__ seg,
                                                         const float* __restrict__ part, float* __restrict__ dE) {
  const int64_t p = blockIdx.x;
  if (seg[p] != p) return;
  const uint64_t v = keys[p] >> 32;
  if (v >= (uint64_t)V || !(p + kChunk < T && (keys[p + kChunk] >> 32) == v)) return;
  int64_t nc = 2;
  while (p + nc * kChunk < T && (keys[p + nc * kChunk] >> 32) == v) ++nc;
  for (int64_t k = threadIdx.x; k < d; k += 256) {
    LocalFoldN<20> f;  // up to 2^20 - 1 chunks: T < 2^25
    for (int64_t c = 0; c < nc; ++c) f.push(part[(p + c * kChunk) * d + k]);
    dE[(int64_t)v * d + k] = f.result();
  }
}

__global__ void fill_zero_kernel(int64_t n, float* __restrict__ x) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i < n) x[i] = 0.0f;
}

// scratch: keys (sort_len(T) uint64), seg (T int32), part (T d floats), each 256-byte aligned
size_t embed_bwd_scratch_bytes(int64_t T, int64_t d) {
  const int64_t P = sort_len(T > 0 ? T : 1);
  auto up = [](size_t b) { return (b + 255) & ~size_t(255); };
  return up(sizeof(uint64_t) * (size_t)P) + up(sizeof(int32_t) * (size_t)(T > 0 ? T : 1)) +
         up(sizeof(float) * (size_t)(T > 0 ? T : 1) * (size_t)(d > 0 ? d : 1));
}

hipError_t embed_bwd_launch(int64_t B, int64_t S, int64_t d, const int32_t* win, int64_t win_ld, int64_t V,
                            const float* dx, float* dE, void* scratch, hipStream_t s) {
  const int64_t T = B * S;
  hipLaunchKernelGGL(fill_zero_kernel, dim3(blocks_for(V * d)), dim3(256), 0, s, V * d, dE);
  if (T == 0) return hipGetLastError();
  const int64_t P = sort_len(T);
  auto up = [](size_t b) { return (b + 255) & ~size_t(255); };
  char* base = static_cast<char*>(scratch);
  uint64_t* keys = reinterpret_cast<uint64_t*>(base);
  int32_t* seg = reinterpret_cast<int32_t*>(base + up(sizeof(uint64_t) * (size_t)P));
  float* part = reinterpret_cast<float*>(base + up(sizeof(uint64_t) * (size_t)P) + up(sizeof(int32_t) * (size_t)T));
  hipLaunchKernelGGL(embed_keys_kernel, dim3(blocks_for(P)), dim3(256), 0, s, T, P, S, win, win_ld, keys);
  const int64_t blk = P < kSortBlk ? P : kSortBlk;
  hipLaunchKernelGGL(bitonic_local_kernel, dim3((unsigned)(P / blk)), dim3(1024), 0, s, keys, blk, (int64_t)0);
  for (int64_t k = 2 * blk; k <= P; k <<= 1) {
    for (int64_t j = k / 2; j >= blk; j >>= 1)
      hipLaunchKernelGGL(bitonic_global_kernel, dim3(blocks_for(P / 2)), dim3(256), 0, s, keys, P, k, j);
    hipLaunchKernelGGL(bitonic_local_kernel, dim3((unsigned)(P / blk)), dim3(1024), 0, s, keys, blk, k);
  }
  hipLaunchKernelGGL(embed_segstart_kernel, dim3(1), dim3(1024), 0, s, T, keys, seg);
  const bool vec = d % 4 == 0 && ((uintptr_t)dx & 15) == 0 && ((uintptr_t)dE & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(embed_chunk_kernel<true>, dim3((unsigned)T), dim3(256), 0, s, T, d, V, keys, seg, dx, dE, part);
  else
    hipLaunchKernelGGL(embed_chunk_kernel<false>, dim3((unsigned)T), dim3(256), 0, s, T, d, V, keys, seg, dx, dE, part);
  hipLaunchKernelGGL(embed_fold_kernel, dim3((unsigned)T), dim3(256), 0, s, T, d, V, keys, seg, part, dE);
  return hipGetLastError();
}

template <int DT>
__global__ void quantize_kernel(int64_t rows, int64_t cols, const void* __restrict__ x,
                                const float* __restrict__ scale, int32_t per_row, int8_t* __restrict__ q) {
  const int64_t n = rows * cols;
  if (!per_row) {  // one step for every value: its reciprocal once per thread
    const float sv = step_daz(scale[0]);
    const bool recip = recip_step_ok(sv);
    const float rs = recip ? 1.0f / sv : 0.0f;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
      const float v = DT == 0 ? static_cast<const float*>(x)[i] : bf16_to_f32(static_cast<const uint16_t*>(x)[i]);
      q[i] = recip ? quant_recip(v, sv, rs) : quant1(v, sv);
    }
    return;
  }
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    const float sv = step_daz(scale[i / cols]);
    const float v = DT == 0 ? static_cast<const float*>(x)[i] : bf16_to_f32(static_cast<const uint16_t*>(x)[i]);
    q[i] = quant1(v, sv);
  }
}

// one step for the whole tensor, fp32 input, 16-byte aligned x and 4-byte aligned q: 4 values per thread
__global__ void quantize_tensor4_kernel(int64_t n, const float* __restrict__ x, const float* __restrict__ scale,
                                        int8_t* __restrict__ q) {
  const float sv = step_daz(scale[0]);
  const bool recip = recip_step_ok(sv);
  const float rs = recip ? 1.0f / sv : 0.0f;
  auto qz = [&](float v) -> uint32_t { return (uint8_t)(recip ? quant_recip(v, sv, rs) : quant1(v, sv)); };
  const int64_t n4 = n >> 2;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
    const float4 v = reinterpret_cast<const float4*>(x)[i];
    reinterpret_cast<uint32_t*>(q)[i] = qz(v.x) | (qz(v.y) << 8) | (qz(v.z) << 16) | (qz(v.w) << 24);
  }
  const int64_t t = n4 * 4 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t < n) q[t] = (int8_t)qz(x[t]);
}

// one step for the whole tensor, bf16 input, 16-byte aligned x and 8-byte aligned q: 8 values per thread
__global__ void quantize_tensor_bf16x8_kernel(int64_t n, const uint16_t* __restrict__ x,
                                              const float* __restrict__ scale, int8_t* __restrict__ q) {
  const float sv = step_daz(scale[0]);
  const bool recip = recip_step_ok(sv);
  const float rs = recip ? 1.0f / sv : 0.0f;
  auto qz = [&](float v) -> uint32_t { return (uint8_t)(recip ? quant_recip(v, sv, rs) : quant1(v, sv)); };
  const int64_t n8 = n >> 3;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n8; i += (int64_t)gridDim.x * 256) {
    const uint4 h = reinterpret_cast<const uint4*>(x)[i];
    const uint32_t w[4] = {h.x, h.y, h.z, h.w};
    uint32_t o[2];
#pragma unroll
    for (int k = 0; k < 2; ++k)
      o[k] = qz(__uint_as_float(w[2 * k] << 16)) | (qz(__uint_as_float(w[2 * k] & 0xFFFF0000u)) << 8) |
             (qz(__uint_as_float(w[2 * k + 1] << 16)) << 16) | (qz(__uint_as_float(w[2 * k + 1] & 0xFFFF0000u)) << 24);
    reinterpret_cast<uint2*>(q)[i] = make_uint2(o[0], o[1]);
  }
  const int64_t t = n8 * 8 + (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (t < n) q[t] = (int8_t)qz(bf16_to_f32(x[t]));
}

// one step per row, bf16 input with 16-byte aligned rows (cols a multiple of 8) and 8-byte aligned q: a
// workgroup per row (grid-stride over rows), 8 values per thread per pass over the row
__global__ __launch_bounds__(256) void quantize_rows_bf16x8_kernel(int64_t rows, int64_t cols,
                                                                   const uint16_t* __restrict__ x,
                                                                   const float* __restrict__ scale,
                                                                   int8_t* __restrict__ q) {
  const int64_t g8 = cols >> 3;
  for (int64_t r = blockIdx.x; r < rows; r += gridDim.x) {
    const float sv = step_daz(scale[r]);
    const uint4* xr = reinterpret_cast<const uint4*>(x + r * cols);
    uint2* qr = reinterpret_cast<uint2*>(q + r * cols);
    for (int64_t i = threadIdx.x; i < g8; i += 256) {
      const uint4 h = xr[i];
      const uint32_t w[4] = {h.x, h.y, h.z, h.w};
      uint32_t o[2];
#pragma unroll
      for (int k = 0; k < 2; ++k)
        o[k] = (uint32_t)(uint8_t)quant1(__uint_as_float(w[2 * k] << 16), sv) |
               ((uint32_t)(uint8_t)quant1(__uint_as_float(w[2 * k] & 0xFFFF0000u), sv) << 8) |
               ((uint32_t)(uint8_t)quant1(__uint_as_float(w[2 * k + 1] << 16), sv) << 16) |
               ((uint32_t)(uint8_t)quant1(__uint_as_float(w[2 * k + 1] & 0xFFFF0000u), sv) << 24);
      qr[i] = make_uint2(o[0], o[1]);
    }
  }
}

hipError_t quantize_launch(int64_t rows, int64_t cols, int32_t dtype, const void* x, const float* scale,
                           int32_t per_row, int8_t* q, hipStream_t s) {
  const int64_t n = rows * cols;
  if (n == 0) return hipSuccess;
  if (dtype == 0 && !per_row && ((uintptr_t)x & 15) == 0 && ((uintptr_t)q & 3) == 0) {
    int64_t b = ((n >> 2) + 255) / 256;
    if (b < 1) b = 1;
    const unsigned grid = (unsigned)(b < (1 << 20) ? b : (1 << 20));
    hipLaunchKernelGGL(quantize_tensor4_kernel, dim3(grid), dim3(256), 0, s, n, (const float*)x, scale, q);
    return hipGetLastError();
  }
  if (dtype == 1 && per_row && cols % 8 == 0 && ((uintptr_t)x & 15) == 0 && ((uintptr_t)q & 7) == 0) {
    const unsigned grid = (unsigned)(rows < 8192 ? rows : 8192);
    hipLaunchKernelGGL(quantize_rows_bf16x8_kernel, dim3(grid), dim3(256), 0, s, rows, cols, (const uint16_t*)x, scale,
                       q);
    return hipGetLastError();
  }
  if (dtype == 1 && !per_row && ((uintptr_t)x & 15) == 0 && ((uintptr_t)q & 7) == 0) {
    int64_t b = ((n >> 3) + 255) / 256;
    if (b < 1) b = 1;
    const unsigned grid = (unsigned)(b < (1 << 20) ? b : (1 << 20));
    hipLaunchKernelGGL(quantize_tensor_bf16x8_kernel, dim3(grid), dim3(256), 0, s, n, (const uint16_t*)x, scale, q);
    return hipGetLastError();
  }
  int64_t b = (n + 255) / 256;
  const unsigned grid = (unsigned)(b < (1 << 20) ? b : (1 << 20));
  if (dtype == 0)
    hipLaunchKernelGGL(quantize_kernel<0>, dim3(grid), dim3(256), 0, s, rows, cols, x, scale, per_row, q);
  else
    hipLaunchKernelGGL(quantize_kernel<1>, dim3(grid), dim3(256), 0, s, rows, cols, x, scale, per_row, q);
  return hipGetLastError();
}

// ---- device evaluation of the primitives -----------------------------------------------------------
__global__ void devmath_kernel(int32_t op, int64_t n, const float* __restrict__ a, const float* __restrict__ b,
                               const float* __restrict__ c, float* __restrict__ out) {
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= n) return;
  float x = a[i], r = 0.0f;
  switch (op) {
    case 0: r = x + b[i]; break;
    case 1: r = x - b[i]; break;
    case 2: r = x * b[i]; break;
    case 3: r = __builtin_fmaf(x, b[i], c[i]); break;
    case 4: r = x / b[i]; break;
    case 5: r = __builtin_sqrtf(x); break;
    case 6: r = cexp(x); break;
    case 7: r = clog(x); break;
    case 8: r = csigmoid(x); break;
    case 9: r = csilu(x); break;
    case 10: r = bf16_to_f32(f32_to_bf16(x)); break;
  }
  out[i] = r;
}

hipError_t devmath_launch(int32_t op, int64_t n, const float* a, const float* b, const float* c, float* out,
                          hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(devmath_kernel, dim3(blocks_for(n)), dim3(256), 0, s, op, n, a, b, c, out);
  return hipGetLastError();
}

}  // namespace canon
