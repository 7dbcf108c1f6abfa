// lsq.hip - the gradient of a learned per-tensor activation step of the int8 projections (R19: the paper's
// int8 quantisation-aware training with learned step-size quantisation for activations).
//
// g_s = RN(R1 over the flat index of RN(dx * delta) * gamma), gamma = RN32(1/sqrt(127 K)) (LSQ's gradient
// scale for K features, computed by the caller), where for each element with v = RN(x / s): delta = -128 below
// the integer range, 127 above it, RN(rne(v) - v) inside; 0 when the step is not > 0 once flushed or v is NaN.
// Pass 1: one workgroup per aligned block of 1024 chunks (a complete subtree of the padded tree); each
// wavefront forms 64 chunks of terms at a time from coalesced loads, stages them transposed in LDS so that
// lane c runs chunk c's chain, and folds the lanes with the pass-through rule.  Pass 2: one workgroup folds
// the block sums (each thread a complete subtree of consecutive sums, then across threads) and scales.
#include <hip/hip_runtime.h>

#include <mutex>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

namespace {

constexpr int kSegs = 4;                        // segments of 64 chunks per wavefront
constexpr int kWaveChunks = 64 * kSegs;         // 256 chunks per wavefront
constexpr int kBlockChunks = 4 * kWaveChunks;   // 1024 chunks (32768 terms) per workgroup
constexpr int kSegTerms = 64 * kChunk;          // 2048 terms per segment

struct Stage {
  float t[64][33];
};

__device__ __forceinline__ float lsq_delta(float x, float s, bool valid) {
  if (!valid) return 0.0f;
  const float v = x / s;  // correctly rounded
  if (!(v == v)) return 0.0f;
  if (v < -128.0f) return -128.0f;
  if (v > 127.0f) return 127.0f;
  return __builtin_rintf(v) - v;  // exact: |rne(v) - v| <= 1/2 (Sterbenz)
}

// terms j .. j+3 (VEC: one 16-byte load of dx and 8 bytes of x; the caller guarantees alignment and that the
// group lies inside [0, n))
template <bool VEC>
__device__ __forceinline__ void terms4(const uint16_t* __restrict__ x, const float* __restrict__ dx, int64_t n,
                                       int64_t j, float s, bool valid, float (&t)[4]) {
  if (VEC && j + 4 <= n) {
    const float4 g = *reinterpret_cast<const float4*>(dx + j);
    const uint2 h = *reinterpret_cast<const uint2*>(x + j);
    t[0] = g.x * lsq_delta(bf16_to_f32((uint16_t)(h.x & 0xFFFFu)), s, valid);
    t[1] = g.y * lsq_delta(bf16_to_f32((uint16_t)(h.x >> 16)), s, valid);
    t[2] = g.z * lsq_delta(bf16_to_f32((uint16_t)(h.y & 0xFFFFu)), s, valid);
    t[3] = g.w * lsq_delta(bf16_to_f32((uint16_t)(h.y >> 16)), s, valid);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      t[i] = (j + i < n) ? dx[j + i] * lsq_delta(bf16_to_f32(x[j + i]), s, valid) : 0.0f;
  }
}

template <bool VEC>
__global__ __launch_bounds__(256) void lsq_block_kernel(int64_t n, const uint16_t* __restrict__ x,
                                                        const float* __restrict__ dx, const float* __restrict__ sp,
                                                        float* __restrict__ part) {
  constexpr int Q = kSegTerms / (64 * 4);  // 4-term groups per lane per segment
  __shared__ Stage st[4];
  __shared__ float wsum[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const float s = step_daz(*sp);
  const bool valid = s > 0.0f;
  const int64_t nc = (n + kChunk - 1) / kChunk;
  const int64_t cw = (int64_t)blockIdx.x * kBlockChunks + (int64_t)w * kWaveChunks;  // wave's first chunk
  LocalFoldN<8> wf;
  for (int sg = 0; sg < kSegs; ++sg) {
    const int64_t c0 = cw + 64 * sg;
    if (c0 >= nc) break;
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int local = 256 * q + 4 * lane;
      float t[4];
      terms4<VEC>(x, dx, n, c0 * kChunk + local, s, valid, t);
      float* dst = &st[w].t[local >> 5][local & 31];
#pragma unroll
      for (int i = 0; i < 4; ++i) dst[i] = t[i];
    }
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
    float p = 0.0f;
    const int64_t c = c0 + lane;
    if (c < nc) {
      const int k1 = (int)(n - c * kChunk < kChunk ? n - c * kChunk : kChunk);
      for (int i = 0; i < k1; ++i) p = p + st[w].t[lane][i];
    }
    const int64_t real = nc - c0;
    const float seg = wave_fold(p, real > 64 ? 64 : (int)real);
    if (lane == 0) wf.push(seg);
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
  }
  if (lane == 0) wsum[w] = wf.result();
  __syncthreads();
  if (threadIdx.x == 0) {  // the four waves: pairs of complete subtrees, a right one without real chunks passed over
    const int64_t cb = (int64_t)blockIdx.x * kBlockChunks;
    float a = wsum[0];
    if (cb + kWaveChunks < nc) a = a + wsum[1];
    if (cb + 2 * kWaveChunks < nc) {
      float b = wsum[2];
      if (cb + 3 * kWaveChunks < nc) b = b + wsum[3];
      a = a + b;
    }
    part[blockIdx.x] = a;
  }
}

// Algorithm 2 over the block sums: thread t folds the aligned run [t G, t G + G) of consecutive sums (a
// complete subtree, G a power of two), then the threads fold with the pass-through rule; times gamma.
__global__ __launch_bounds__(256) void lsq_final_kernel(int64_t nparts, const float* __restrict__ part, float gamma,
                                                        float* __restrict__ out) {
  const int64_t G = block_chunks(nparts, 256);
  const int64_t b0 = (int64_t)threadIdx.x * G;
  LocalFoldN<16> f;
  for (int64_t i = b0; i < b0 + G && i < nparts; ++i) f.push(part[i]);
  const float p = f.result();
  const int64_t nthr = (nparts + G - 1) / G;
  const float total = block_fold(p, nthr);
  if (threadIdx.x == 0) out[0] = total * gamma;
}

}  // namespace

int64_t lsq_grad_parts(int64_t n) { return (n + (int64_t)kBlockChunks * kChunk - 1) / ((int64_t)kBlockChunks * kChunk); }

// ---- the allocation-free variant: the block sums live in a file-scope device array ----
// One copy per GPU, held until the process ends.  Host code never uses the array's name as an address:
// the device address of each GPU's copy comes from hipGetSymbolAddress with that GPU current.
constexpr int64_t kScratchParts = 65536;  // 256 KiB: block sums of up to 2^31 terms
static __device__ __align__(256) float scratch[kScratchParts];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static float* g_scratch_dev[kMaxDevices];  // device address of the current GPU's copy, set on first use

int64_t lsq_noalloc_max_terms() { return kScratchParts * (int64_t)kBlockChunks * kChunk; }

hipError_t lsq_scratch(float** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return e != hipSuccess ? e : hipErrorInvalidSymbol;
    g_scratch_dev[dev] = static_cast<float*>(ptr);
  }
  *out = g_scratch_dev[dev];
  return hipSuccess;
}

hipError_t lsq_grad_launch(int64_t n, const uint16_t* x, const float* s, const float* dx, float gamma, float* part,
                           float* out, hipStream_t st) {
  const int64_t nparts = lsq_grad_parts(n);
  if (nparts == 0) {
    hipLaunchKernelGGL(lsq_final_kernel, dim3(1), dim3(256), 0, st, (int64_t)0, part, gamma, out);
    return hipGetLastError();
  }
  const bool vec = n % 4 == 0 && ((uintptr_t)x & 7) == 0 && ((uintptr_t)dx & 15) == 0;
  if (vec) hipLaunchKernelGGL(lsq_block_kernel<true>, dim3((unsigned)nparts), dim3(256), 0, st, n, x, dx, s, part);
  else hipLaunchKernelGGL(lsq_block_kernel<false>, dim3((unsigned)nparts), dim3(256), 0, st, n, x, dx, s, part);
  hipLaunchKernelGGL(lsq_final_kernel, dim3(1), dim3(256), 0, st, nparts, part, gamma, out);
  return hipGetLastError();
}

}  // namespace canon
