// optim.hip - the gradient plan (R7: Algorithm 1 with Algorithm 2 over replicas) and AdamW (R9).
// All of these are streaming, HBM-bound kernels: one element per thread, no cross-element arithmetic, so
// the order of every per-element operation is fixed by the code and independent of the launch shape.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

static inline unsigned grid_for(int64_t n) {
  int64_t b = (n + 255) / 256;
  return (unsigned)(b < 65536 * 16 ? b : 65536 * 16);  // grid-stride beyond this
}

// Algorithm 1 for one element with its buffers' values in v[0..NB): rank r's microbatches are v[r*accum ..
// r*accum + accum), ranks in mesh order (shard index fastest).  Each microbatch gradient is scaled by
// RN(1/accum) and summed from +0; ranks of one replica are summed in ascending shard order and scaled by
// RN(1/dp_shard); the replica partials go through Algorithm 2's binary-carry stack (earlier block on the
// left, Result from the lowest level up) and the total is scaled by RN(1/dp_replicate).  The loop over the
// buffers is unrolled with constant indices, so v stays in registers; the branches depend only on the plan.
template <int NB>
__device__ __forceinline__ float plan_element(const float (&v)[NB], int accum, int dp_shard, float inv_accum,
                                              float inv_shard, float inv_rep) {
  float stack[8];
  int pushed = 0;
  float g = 0.0f, inner = 0.0f;
  int k = 0, shard = 0;
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    g = ((k == 0) ? 0.0f : g) + v[b] * inv_accum;
    if (++k == accum) {
      k = 0;
      inner = (shard == 0) ? g : inner + g;
      if (++shard == dp_shard) {
        shard = 0;
        float part = inner * inv_shard;
#pragma unroll
        for (int L = 0; L < 8; ++L) {
          if ((pushed >> L) & 1) {
            part = stack[L] + part;
          } else {
            stack[L] = part;
            break;
          }
        }
        ++pushed;
      }
    }
  }
  float res = 0.0f;
  bool have = false;
#pragma unroll
  for (int L = 0; L < 8; ++L) {
    if ((pushed >> L) & 1) {
      if (!have) {
        res = stack[L];
        have = true;
      } else {
        res = stack[L] + res;
      }
    }
  }
  return res * inv_rep;
}

// NB buffers known at compile time: four elements per thread with 16-byte streaming loads, all NB loads
// issued before the arithmetic; the n % 4 tail is done by the first threads of the grid.
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <int NB>
__global__ __launch_bounds__(256) void grad_accum_vec_kernel(int accum, int dp_shard, int64_t n, PlanPtrs ptrs,
                                                             float inv_accum, float inv_shard, float inv_rep,
                                                             float* __restrict__ out) {
  const int64_t n4 = n >> 2;
  const int64_t stride = (int64_t)gridDim.x * 256;
  const int64_t tid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (int64_t i = tid; i < n4; i += stride) {
    f32x4 q[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) q[b] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(ptrs.p[b]) + i);
    f32x4 r;
    {
      float v[NB];
#pragma unroll
      for (int b = 0; b < NB; ++b) v[b] = q[b].x;
      r.x = plan_element<NB>(v, accum, dp_shard, inv_accum, inv_shard, inv_rep);
#pragma unroll
      for (int b = 0; b < NB; ++b) v[b] = q[b].y;
      r.y = plan_element<NB>(v, accum, dp_shard, inv_accum, inv_shard, inv_rep);
#pragma unroll
      for (int b = 0; b < NB; ++b) v[b] = q[b].z;
      r.z = plan_element<NB>(v, accum, dp_shard, inv_accum, inv_shard, inv_rep);
#pragma unroll
      for (int b = 0; b < NB; ++b) v[b] = q[b].w;
      r.w = plan_element<NB>(v, accum, dp_shard, inv_accum, inv_shard, inv_rep);
    }
    __builtin_nontemporal_store(r, reinterpret_cast<f32x4*>(out) + i);
  }
  const int64_t t = n4 * 4 + tid;
  if (t < n) {
    float v[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) v[b] = ptrs.p[b][t];
    out[t] = plan_element<NB>(v, accum, dp_shard, inv_accum, inv_shard, inv_rep);
  }
}

// Any plan up to kMaxFusedBuffers buffers, one element per thread (the same walk as plan_element, with the
// buffers read as the walk reaches them).
__global__ __launch_bounds__(256) void grad_accum_fused_kernel(int accum, int dp_shard, int dp_replicate, int64_t n,
                                                               PlanPtrs ptrs, float inv_accum, float inv_shard,
                                                               float inv_rep, float* __restrict__ out) {
  const int N = dp_shard * dp_replicate;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    float stack[8];
    int pushed = 0;
    float inner = 0.0f;
    for (int r = 0; r < N; ++r) {
      float g = 0.0f;
      for (int k = 0; k < accum; ++k) g = g + ptrs.p[r * accum + k][i] * inv_accum;
      const int shard = r % dp_shard;
      inner = (shard == 0) ? g : inner + g;
      if (shard == dp_shard - 1) {
        float part = inner * inv_shard;
#pragma unroll
        for (int L = 0; L < 8; ++L) {
          if ((pushed >> L) & 1) {
            part = stack[L] + part;
          } else {
            stack[L] = part;
            break;
          }
        }
        ++pushed;
      }
    }
    float res = 0.0f;
    bool have = false;
#pragma unroll
    for (int L = 0; L < 8; ++L) {
      if ((pushed >> L) & 1) {
        if (!have) {
          res = stack[L];
          have = true;
        } else {
          res = stack[L] + res;
        }
      }
    }
    out[i] = res * inv_rep;
  }
}

hipError_t grad_accum_fused_launch(int accum, int dp_shard, int dp_replicate, int64_t n, const PlanPtrs& ptrs,
                                   float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const float inv_accum = (float)(1.0 / accum), inv_shard = (float)(1.0 / dp_shard),
              inv_rep = (float)(1.0 / dp_replicate);  // RN32 of each reciprocal
  const int nb = accum * dp_shard * dp_replicate;
  bool aligned = ((uintptr_t)out & 15) == 0;
  for (int b = 0; b < nb; ++b) aligned = aligned && ((uintptr_t)ptrs.p[b] & 15) == 0;
  if (aligned && nb <= 16) {
    int64_t blocks = ((n >> 2) + 255) / 256;
    if (blocks < 1) blocks = 1;
    const unsigned grid = (unsigned)(blocks < (1 << 20) ? blocks : (1 << 20));  // grid-stride beyond 2^20 groups
#define CANON_GA(NBV)                                                                                         \
  case NBV:                                                                                                   \
    hipLaunchKernelGGL(grad_accum_vec_kernel<NBV>, dim3(grid), dim3(256), 0, s, accum, dp_shard, n, ptrs,      \
                       inv_accum, inv_shard, inv_rep, out);                                                   \
    return hipGetLastError();
    switch (nb) {
      CANON_GA(1) CANON_GA(2) CANON_GA(3) CANON_GA(4) CANON_GA(5) CANON_GA(6) CANON_GA(7) CANON_GA(8)
      CANON_GA(9) CANON_GA(10) CANON_GA(11) CANON_GA(12) CANON_GA(13) CANON_GA(14) CANON_GA(15) CANON_GA(16)
      default: break;
    }
#undef CANON_GA
  }
  hipLaunchKernelGGL(grad_accum_fused_kernel, dim3(grid_for(n)), dim3(256), 0, s, accum, dp_shard, dp_replicate, n,
                     ptrs, inv_accum, inv_shard, inv_rep, out);
  return hipGetLastError();
}

__global__ void plan_accum_kernel(int64_t n, const float* __restrict__ grad, float inv, int first, float* out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    float t = grad[i] * inv;
    float base = first ? 0.0f : out[i];
    out[i] = base + t;
  }
}

__global__ void plan_shard_kernel(int64_t n, const float* __restrict__ a, int first, float* out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = first ? a[i] : out[i] + a[i];
}

__global__ void plan_merge_kernel(int64_t n, const float* __restrict__ lower, float* out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = lower[i] + out[i];
}

__global__ void plan_scale_kernel(int64_t n, const float* x, float inv, float* out) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    out[i] = x[i] * inv;
}

// With one microbatch per rank (accum = 1) the rank's sum g_r = RN(+0 + RN(grad * inv_accum)) goes straight
// into the ascending shard sum: inner = g_r on shard 0, RN(inner + g_r) after; on the last shard the result is
// also scaled, RN(inner * inv_shard).  The same operations as plan_accum, plan_shard and plan_scale in turn,
// in one pass over the gradient (16-byte accesses when n % 4 == 0 and both buffers are aligned).
template <bool VEC>
__global__ __launch_bounds__(256) void plan_rank_kernel(int64_t n, const float* __restrict__ grad, float inv_accum,
                                                        int first, int last, float inv_shard, float* __restrict__ inner) {
  auto one = [&](float gv, float iv) -> float {
    const float t = gv * inv_accum;
    const float gr = 0.0f + t;
    float v = first ? gr : iv + gr;
    if (last) v = v * inv_shard;
    return v;
  };
  if (VEC) {
    const int64_t n4 = n >> 2;
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += (int64_t)gridDim.x * 256) {
      const float4 gv = reinterpret_cast<const float4*>(grad)[i];
      float4 iv = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
      if (!first) iv = reinterpret_cast<const float4*>(inner)[i];
      float4 o;
      o.x = one(gv.x, iv.x);
      o.y = one(gv.y, iv.y);
      o.z = one(gv.z, iv.z);
      o.w = one(gv.w, iv.w);
      reinterpret_cast<float4*>(inner)[i] = o;
    }
  } else {
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
      inner[i] = one(grad[i], first ? 0.0f : inner[i]);
  }
}

hipError_t plan_rank_launch(int64_t n, const float* grad, float inv_accum, int first, int last, float inv_shard,
                            float* inner, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const bool vec = n % 4 == 0 && ((uintptr_t)grad & 15) == 0 && ((uintptr_t)inner & 15) == 0;
  if (vec)
    hipLaunchKernelGGL(plan_rank_kernel<true>, dim3(grid_for(n / 4)), dim3(256), 0, s, n, grad, inv_accum, first, last,
                       inv_shard, inner);
  else
    hipLaunchKernelGGL(plan_rank_kernel<false>, dim3(grid_for(n)), dim3(256), 0, s, n, grad, inv_accum, first, last,
                       inv_shard, inner);
  return hipGetLastError();
}

hipError_t plan_accum_launch(int64_t n, const float* grad, float inv, int first, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(plan_accum_kernel, dim3(grid_for(n)), dim3(256), 0, s, n, grad, inv, first, out);
  return hipGetLastError();
}

hipError_t plan_shard_launch(int64_t n, const float* a, int first, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(plan_shard_kernel, dim3(grid_for(n)), dim3(256), 0, s, n, a, first, out);
  return hipGetLastError();
}

hipError_t plan_merge_launch(int64_t n, const float* lower, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(plan_merge_kernel, dim3(grid_for(n)), dim3(256), 0, s, n, lower, out);
  return hipGetLastError();
}

hipError_t plan_scale_launch(int64_t n, const float* x, float inv, float* out, hipStream_t s) {
  if (n == 0) return hipSuccess;
  hipLaunchKernelGGL(plan_scale_kernel, dim3(grid_for(n)), dim3(256), 0, s, n, x, inv, out);
  return hipGetLastError();
}

struct AdamWK {
  float lr, beta1, omb1, beta2, omb2, inv_bc1, inv_bc2, eps, decay_factor;
};

__global__ __launch_bounds__(256) void adamw_kernel(int64_t n, uint16_t* __restrict__ p16, float* __restrict__ m,
                                                    float* __restrict__ v, const float* __restrict__ g, int decay,
                                                    AdamWK k, const float* __restrict__ gscale,
                                                    const int32_t* __restrict__ skip) {
  if (skip && *skip) return;
  const float c = gscale ? *gscale : 1.0f;
  const bool clip = c < 1.0f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256) {
    float p = bf16_to_f32(p16[i]);
    if (decay) p = p * k.decay_factor;
    float gi = g[i];
    if (clip) gi = gi * c;
    float m1 = k.beta1 * m[i];
    float m2 = k.omb1 * gi;
    float mi = m1 + m2;
    float gg = gi * gi;
    float v1 = k.beta2 * v[i];
    float v2 = k.omb2 * gg;
    float vi = v1 + v2;
    float mh = mi * k.inv_bc1;
    float vh = vi * k.inv_bc2;
    float den = __builtin_sqrtf(vh) + k.eps;
    float u = mh / den;
    float step = k.lr * u;
    p = p - step;
    m[i] = mi;
    v[i] = vi;
    p16[i] = f32_to_bf16(p);
  }
}

hipError_t adamw_launch(int64_t n, uint16_t* p, float* m, float* v, const float* g, int decay, const float* c9,
                        const float* gscale, const int32_t* skip_flag, hipStream_t s) {
  if (n == 0) return hipSuccess;
  AdamWK k{c9[0], c9[1], c9[2], c9[3], c9[4], c9[5], c9[6], c9[7], c9[8]};
  hipLaunchKernelGGL(adamw_kernel, dim3(grid_for(n)), dim3(256), 0, s, n, p, m, v, g, decay, k, gscale, skip_flag);
  return hipGetLastError();
}

__global__ void set_nan_if_kernel(const int32_t* flag, float* x) {
  if (*flag) x[0] = __builtin_nanf("");
}

hipError_t set_nan_if_launch(const int32_t* flag, float* x, hipStream_t s) {
  hipLaunchKernelGGL(set_nan_if_kernel, dim3(1), dim3(1), 0, s, flag, x);
  return hipGetLastError();
}

}  // namespace canon
