// norm.hip - the global gradient norm of R15 (the optimizer paragraph's clip to a global l2 norm of 1.0),
// the clip coefficient and spike decision (the section on gradient behaviour: a pre-clip norm above 5
// skips five optimizer steps), and the clip itself.
//
// The gradient tensors laid end to end in the declared order are one vector; its sum of squares is R1 over
// that vector's flat index (chunks of 32 may run across a tensor boundary).  Pass 1: one workgroup per
// aligned block of kNormBlockChunks chunks, i.e. one complete (or, for the last, left-filled) subtree of
// the padded tree; each wavefront reads 64 chunks at a time coalesced, squares on the way in, stages them
// in LDS transposed so that lane c runs chunk c's chain, and folds the lanes with the pass-through rule.
// Pass 2: one workgroup folds the block sums (Algorithm 2 over complete subtrees gives the same tree), takes
// the square root and makes the decisions.  HBM bound: 4 bytes read per gradient element.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

namespace {

constexpr int kWaveSegs = 4;                         // segments of 64 chunks per wavefront
constexpr int kWaveChunks = 64 * kWaveSegs;          // 256 chunks per wavefront
constexpr int kNormBlockChunks = 4 * kWaveChunks;    // 4 wavefronts: 1024 chunks (32768 terms) per workgroup
constexpr int kFinalWaves = 16;                      // wavefronts of the block-sum fold
constexpr int kSegTerms = 64 * kChunk;               // 2048 terms per segment
constexpr float kClipEps = 1e-6f;                    // RN32(1e-6), added to the norm before the division

struct Stage {
  float t[64][33];
};

typedef float f32x4 __attribute__((ext_vector_type(4)));

// W consecutive terms starting at flat index j (W = 4: the host guarantees that a W-group never crosses a
// tensor boundary or the end, and that every tensor base is 16-byte aligned).
template <int W, bool MULTI>
__device__ __forceinline__ void load_terms(const NormSrc& src, int64_t n, int64_t j, int& cur, float (&f)[W]) {
  if (j >= n) {
#pragma unroll
    for (int i = 0; i < W; ++i) f[i] = 0.0f;
    return;
  }
  const float* p;
  if (MULTI) {
    while (j >= src.start[cur + 1]) ++cur;
    p = src.ptr[cur] + (j - src.start[cur]);
  } else {
    p = src.one + j;
  }
  if (W == 4) {
    const f32x4 v = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
    f[0] = v.x; f[1] = v.y; f[2] = v.z; f[3] = v.w;
  } else {
    f[0] = __builtin_nontemporal_load(p);
  }
}

// first tensor whose range holds flat index j (tensors of size 0 are skipped)
__device__ __forceinline__ int find_tensor(const NormSrc& src, int64_t j) {
  int lo = 0, hi = src.nt - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (src.start[mid] <= j) lo = mid; else hi = mid - 1;
  }
  while (lo < src.nt - 1 && src.start[lo + 1] <= j) ++lo;
  return lo;
}

template <int W, bool MULTI>
__global__ __launch_bounds__(256) void gnorm_block_kernel(int64_t n, NormSrc src, float* __restrict__ part) {
  constexpr int Q = kSegTerms / (64 * W);  // W-groups per lane per segment
  __shared__ Stage st[4];
  __shared__ float wsum[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int64_t nc = (n + kChunk - 1) / kChunk;
  const int64_t cw = (int64_t)blockIdx.x * kNormBlockChunks + (int64_t)w * kWaveChunks;  // wave's first chunk
  int cur = 0;
  if (MULTI) cur = find_tensor(src, cw * kChunk + W * lane < n ? cw * kChunk + W * lane : n - 1);
  // the wave's segments are consecutive complete subtrees of 64 chunks: a binary-carry fold over the real
  // ones gives the wave's subtree with the pass-through rule
  LocalFoldN<8> wf;
  float nxt[Q][W];
#pragma unroll
  for (int q = 0; q < Q; ++q) load_terms<W, MULTI>(src, n, cw * kChunk + 64 * W * q + W * lane, cur, nxt[q]);
#pragma unroll
  for (int sg = 0; sg < kWaveSegs; ++sg) {
    const int64_t c0 = cw + 64 * sg;
    if (c0 >= nc) break;
    float f[Q][W];
#pragma unroll
    for (int q = 0; q < Q; ++q)
#pragma unroll
      for (int i = 0; i < W; ++i) f[q][i] = nxt[q][i];
    if (sg + 1 < kWaveSegs) {
#pragma unroll
      for (int q = 0; q < Q; ++q)
        load_terms<W, MULTI>(src, n, (c0 + 64) * kChunk + 64 * W * q + W * lane, cur, nxt[q]);
    }
#pragma unroll
    for (int q = 0; q < Q; ++q) {
      const int local = 64 * W * q + W * lane;
      float* dst = &st[w].t[local >> 5][local & 31];
#pragma unroll
      for (int i = 0; i < W; ++i) dst[i] = f[q][i] * f[q][i];
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
  // the workgroup's four waves: pairs of complete subtrees, the right one passed over when it holds no real
  // chunk
  if (threadIdx.x == 0) {
    const int64_t cb = (int64_t)blockIdx.x * kNormBlockChunks;
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

// Fold of the block sums, square root, clip coefficient, spike counter.  bad (may be null): a set flag
// means the gradient is not valid (an out-of-range token): the norm is NaN, no update is applied and the
// spike counter is left alone.
__global__ __launch_bounds__(64 * kFinalWaves) void gnorm_final_kernel(
    int64_t nb, const float* __restrict__ part, float max_norm, float spike_norm, int32_t skip_steps,
    const int32_t* __restrict__ bad, float* norm_out, float* coef_out, int32_t* skip_state, int32_t* skip_flag,
    int32_t* skipped_out) {
  // wave w folds the aligned range [w R, (w + 1) R) of block sums, R a power of two >= 64: 64 consecutive
  // sums per read (coalesced) folded across the lanes, those 64-subtrees pushed into a binary-carry fold;
  // then the waves' subtrees are folded level by level with the pass-through rule
  __shared__ float wsum[kFinalWaves];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  int64_t R = 64;
  while (kFinalWaves * R < nb) R <<= 1;
  LocalFoldN<24> wf;
  const int64_t r0 = (int64_t)w * R, r1 = (r0 + R < nb) ? r0 + R : nb;
  constexpr int kBatch = 16;
  for (int64_t b = r0; b < r1; b += 64 * kBatch) {
    float v[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int64_t j = b + 64 * i + lane;
      v[i] = j < r1 ? part[j] : 0.0f;
    }
#pragma unroll
    for (int i = 0; i < kBatch; ++i) {
      const int64_t s0 = b + 64 * i;
      if (s0 < r1) {
        const float t = wave_fold(v[i], (int)(r1 - s0 < 64 ? r1 - s0 : 64));
        if (lane == 0) wf.push(t);
      }
    }
  }
  if (lane == 0) wsum[w] = wf.result();
  __syncthreads();
  if (threadIdx.x != 0) return;
  float v[kFinalWaves];
#pragma unroll
  for (int q = 0; q < kFinalWaves; ++q) v[q] = wsum[q];
#pragma unroll
  for (int d = 1; d < kFinalWaves; d <<= 1)
#pragma unroll
    for (int q = 0; q + d < kFinalWaves; q += 2 * d)
      if ((q + d) * R < nb) v[q] = v[q] + v[q + d];
  const float q = v[0];
  float norm = __builtin_sqrtf(q);
  float coef;
  int32_t skip;
  if (bad && *bad) {
    norm = __builtin_nanf("");
    coef = 1.0f;
    skip = 1;
  } else {
    const float den = norm + kClipEps;
    coef = max_norm / den;
    int32_t left = skip_state ? *skip_state : 0;
    if (skip_steps > 0 && !(norm <= spike_norm)) left = skip_steps;
    skip = left > 0;
    if (skip) left -= 1;
    if (skip_state) *skip_state = left;
  }
  if (norm_out) *norm_out = norm;
  *coef_out = coef;
  if (skip_flag) *skip_flag = skip;
  if (skipped_out) *skipped_out = skip;
}

// g <- RN(g * coef) when coef < 1
template <int W>
__global__ __launch_bounds__(256) void clip_scale_kernel(int64_t n, float* __restrict__ g,
                                                         const float* __restrict__ coef) {
  const float c = *coef;
  if (!(c < 1.0f)) return;
  const int64_t nv = n / W;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < nv; i += (int64_t)gridDim.x * 256) {
    if (W == 4) {
      float4 v = reinterpret_cast<float4*>(g)[i];
      v.x = v.x * c; v.y = v.y * c; v.z = v.z * c; v.w = v.w * c;
      reinterpret_cast<float4*>(g)[i] = v;
    } else {
      g[i] = g[i] * c;
    }
  }
  if (W == 4 && blockIdx.x == 0 && threadIdx.x < (n & 3)) g[4 * nv + threadIdx.x] = g[4 * nv + threadIdx.x] * c;
}

inline bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

}  // namespace

int64_t gnorm_blocks(int64_t n) {
  const int64_t nc = (n + kChunk - 1) / kChunk;
  return (nc + kNormBlockChunks - 1) / kNormBlockChunks;
}

hipError_t gnorm_launch(const NormSrc& src, int64_t n, int vec4, float* part, const ClipDecision& d, hipStream_t s) {
  const int64_t nb = gnorm_blocks(n);
  if (nb > 0x7fffffff) return hipErrorInvalidValue;
  if (nb > 0) {
    const dim3 grid((unsigned)nb), block(256);
    if (src.nt == 0 || src.one) {
      if (vec4) hipLaunchKernelGGL((gnorm_block_kernel<4, false>), grid, block, 0, s, n, src, part);
      else hipLaunchKernelGGL((gnorm_block_kernel<1, false>), grid, block, 0, s, n, src, part);
    } else {
      if (vec4) hipLaunchKernelGGL((gnorm_block_kernel<4, true>), grid, block, 0, s, n, src, part);
      else hipLaunchKernelGGL((gnorm_block_kernel<1, true>), grid, block, 0, s, n, src, part);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(gnorm_final_kernel, dim3(1), dim3(64 * kFinalWaves), 0, s, nb, part, d.max_norm, d.spike_norm, d.skip_steps,
                     d.bad, d.norm_out, d.coef_out, d.skip_state, d.skip_flag, d.skipped_out);
  return hipGetLastError();
}

hipError_t clip_scale_launch(int64_t n, float* g, const float* coef, hipStream_t s) {
  if (n == 0) return hipSuccess;
  const bool v4 = al16(g);
  const int64_t units = v4 ? n / 4 : n;
  int64_t blocks = (units + 255) / 256;
  if (blocks < 1) blocks = 1;
  if (blocks > 65536) blocks = 65536;
  if (v4) hipLaunchKernelGGL(clip_scale_kernel<4>, dim3((unsigned)blocks), dim3(256), 0, s, n, g, coef);
  else hipLaunchKernelGGL(clip_scale_kernel<1>, dim3((unsigned)blocks), dim3(256), 0, s, n, g, coef);
  return hipGetLastError();
}

}  // namespace canon
