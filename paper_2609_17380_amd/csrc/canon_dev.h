// canon_dev.h - device-side numerics of CANON-v1 for gfx950.
//
// R0 (binary32, round to nearest even, subnormals flushed) is what gfx950 computes natively in flush mode:
// this library is built with -fgpu-flush-denormals-to-zero, so every VALU and MFMA operation reads
// subnormal inputs as signed zero and flushes a result whose rounding to 24 bits with unbounded exponent
// is below 2^-126 (IEEE tininess after rounding).  Division and square root are the compiler's correctly
// rounded sequences (-fhip-fp32-correctly-rounded-divide-sqrt).  -ffp-contract=off keeps every multiply
// and add a separate rounding unless written as __builtin_fmaf.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace canon {

constexpr int kChunk = 32;

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  // exact widening; a subnormal bf16 is read as zero of its sign (R0 input rule)
  uint32_t u = (uint32_t)h << 16;
  if ((u & 0x7F800000u) == 0u) u &= 0x80000000u;
  return __uint_as_float(u);
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  // a subnormal input reads as zero of its sign; then round to nearest even on the 16 dropped bits
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7F800000u) == 0u) u &= 0x80000000u;
  u = u + 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ---- cexp: Cody-Waite reduction by ln 2 (two parts), degree-7 Taylor polynomial (Horner, separate
// multiply and add), exact scaling by 2^k.  Constants are the binary32 roundings of their definitions.
constexpr float kLog2e = 0x1.715476p+0f;        // RN32(1/ln 2)              0x3FB8AA3B
constexpr float kLn2Hi = 0x1.62e4p-1f;          // ln 2 cut to 15 bits       0x3F317200
constexpr float kLn2Lo = 0x1.7f7d1cp-20f;       // RN32(ln 2 - kLn2Hi)       0x35BFBE8E
constexpr float kInvFact2 = 0x1p-1f;            // 1/2!
constexpr float kInvFact3 = 0x1.555556p-3f;     // RN32(1/3!)                0x3E2AAAAB
constexpr float kInvFact4 = 0x1.555556p-5f;     // RN32(1/4!)                0x3D2AAAAB
constexpr float kInvFact5 = 0x1.111112p-7f;     // RN32(1/5!)                0x3C088889
constexpr float kInvFact6 = 0x1.6c16c2p-10f;    // RN32(1/6!)                0x3AB60B61
constexpr float kInvFact7 = 0x1.a01a02p-13f;    // RN32(1/7!)                0x39500D01

__device__ __forceinline__ float cexp(float x) {
  // written without branches (the range checks select the result), so unrolled loops of cexp stay
  // straight-line code; the arithmetic is the same sequence of roundings either way
  float t = x * kLog2e;
  float kf = __builtin_rintf(t);  // nearest integer, ties to even
  float hi = kf * kLn2Hi;
  float lo = kf * kLn2Lo;
  float r = x - hi;
  r = r - lo;
  float p = kInvFact7;
  p = p * r; p = p + kInvFact6;
  p = p * r; p = p + kInvFact5;
  p = p * r; p = p + kInvFact4;
  p = p * r; p = p + kInvFact3;
  p = p * r; p = p + kInvFact2;
  p = p * r; p = p + 1.0f;
  p = p * r; p = p + 1.0f;
  const float kc = fminf(fmaxf(kf, -126.0f), 127.0f);  // k itself whenever the result is not selected away
  const int k = (int)kc;
  float scale = __uint_as_float((uint32_t)(k + 127) << 23);
  float res = p * scale;
  res = (kf < -125.0f) ? 0.0f : res;
  res = (kf > 127.0f) ? __builtin_inff() : res;
  return res;
}

// ---- clog: x = 2^e f, f in (sqrt(1/2), sqrt(2)]; s = (f-1)/(f+1); log f = 2 atanh(s) by the odd series
// through s^11; result = e*ln2 (two parts) + log f.
constexpr float kSqrt2 = 0x1.6a09e6p+0f;        // RN32(sqrt 2)              0x3FB504F3
constexpr float kInv3 = 0x1.555556p-2f;         // RN32(1/3)                 0x3EAAAAAB
constexpr float kInv5 = 0x1.99999ap-3f;         // RN32(1/5)                 0x3E4CCCCD
constexpr float kInv7 = 0x1.24924ap-3f;         // RN32(1/7)                 0x3E124925
constexpr float kInv9 = 0x1.c71c72p-4f;         // RN32(1/9)                 0x3DE38E39
constexpr float kInv11 = 0x1.745d18p-4f;        // RN32(1/11)                0x3DBA2E8C

__device__ __forceinline__ float clog(float x) {
  uint32_t u = __float_as_uint(x);
  if ((u & 0x7F800000u) == 0u) return -__builtin_inff();  // zero or subnormal (read as zero)
  if (u & 0x80000000u) return __builtin_nanf("");
  if ((u & 0x7F800000u) == 0x7F800000u) return x;
  int e = (int)((u >> 23) & 0xFFu) - 127;
  float f = __uint_as_float((u & 0x7FFFFFu) | 0x3F800000u);
  if (f > kSqrt2) {
    f = f * 0.5f;
    e += 1;
  }
  float num = f - 1.0f;
  float den = f + 1.0f;
  float s = num / den;
  float z = s * s;
  float q = kInv11;
  q = q * z; q = q + kInv9;
  q = q * z; q = q + kInv7;
  q = q * z; q = q + kInv5;
  q = q * z; q = q + kInv3;
  q = q * z; q = q + 1.0f;
  float s2 = s + s;
  float lf = s2 * q;
  float ef = (float)e;
  float a = ef * kLn2Lo;
  a = a + lf;
  float b = ef * kLn2Hi;
  return b + a;
}

__device__ __forceinline__ float csigmoid(float x) {
  float e = cexp(-x);
  float den = 1.0f + e;
  return 1.0f / den;
}

__device__ __forceinline__ float csilu(float x) { return x * csigmoid(x); }

// Quantiser of the int8 quantised linear: q = clamp(rne(RN(x / s)), -128, 127), x fp32 (dtype 0) or bf16
// (dtype 1), one step per row or for the whole tensor.  A step that is not > 0 once flushed, or a NaN
// quotient, gives 0.
__device__ __forceinline__ int8_t quant1(float v, float sv) {
  int8_t out = 0;
  if (sv > 0.0f) {
    const float t = v / sv;
    if (t == t) {
      const float r = __builtin_rintf(t);
      out = (int8_t)(int)fminf(fmaxf(r, -128.0f), 127.0f);
    }
  }
  return out;
}

// The same quantiser through the reciprocal of a step shared by many values: for a step s in (0, 2^126]
// (positive, normal, with a normal reciprocal) and rs = RN(1/s), t = RN(v * rs) lies within |v/s| 2^-23
// (1 + 2^-25) of v/s.  |t| >= 129 means |v/s| > 128.9: the clamp decides.  Otherwise |t - v/s| < 1.6e-5 and
// |RN(v/s) - v/s| <= 2^-17, so when t is farther than 2^-15 from every half-integer no rounding boundary
// separates t from RN(v/s) and both round to the same integer; closer than that, the correctly rounded
// quotient decides.  A NaN t falls through to it as well.
__device__ __forceinline__ bool recip_step_ok(float s) { return s > 0.0f && s <= 0x1p126f; }

__device__ __forceinline__ int8_t quant_recip(float v, float s, float rs) {
  const float t = v * rs;
  if (fabsf(t) >= 129.0f) return t > 0.0f ? (int8_t)127 : (int8_t)-128;
  const float n = __builtin_rintf(t);
  const float d = fabsf(t - n);  // exact (Sterbenz), at most 1/2
  if (0.5f - d > 0x1p-15f) return (int8_t)(int)fminf(fmaxf(n, -128.0f), 127.0f);
  return quant1(v, s);
}

__device__ __forceinline__ float step_daz(float s) {
  uint32_t sb = __float_as_uint(s);
  if ((sb & 0x7F800000u) == 0u) sb &= 0x80000000u;  // a subnormal step reads as zero
  return __uint_as_float(sb);
}

// ---- R1 helpers ---------------------------------------------------------------------------------
// Algorithm 2 over nparts chunk partials held one per lane of a wavefront (lane = chunk index, lanes
// >= nparts ignored): level by level, a node adds its right neighbour's subtree only when that subtree
// holds at least one real chunk, otherwise it passes through unchanged.  This is the zero-padded perfect
// tree without adding any padding, i.e. the binary-carry fold with leftover blocks combined smallest
// first.  Returns the total in lane 0.
__device__ __forceinline__ float wave_fold(float p, int nparts) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int s = 1; s < 64; s <<= 1) {
    float other = __shfl_down(p, s, 64);
    if ((lane & (2 * s - 1)) == 0 && lane + s < nparts) p = p + other;
  }
  return p;
}

// Binary-carry fold of a lane's consecutive chunk partials (Algorithm 2 on one lane): up to 2^LEVELS - 1
// pushes.
template <int LEVELS>
struct LocalFoldN {
  float s[LEVELS];
  int64_t count = 0;
  __device__ void push(float p) {
#pragma unroll
    for (int L = 0; L < LEVELS; ++L) {
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
    for (int L = 0; L < LEVELS; ++L) {
      if ((count >> L) & 1) {
        if (!have) {
          r = s[L];
          have = true;
        } else {
          r = s[L] + r;
        }
      }
    }
    return r;
  }
};
using LocalFold = LocalFoldN<16>;  // a lane block of up to 2^16 - 1 chunks

// chunks per lane so that `lanes` lanes cover nc chunks with aligned power-of-two blocks
__device__ __forceinline__ int64_t block_chunks(int64_t nc, int lanes) {
  int64_t G = 1;
  while (G * lanes < nc) G <<= 1;
  return G;
}

// Fold of per-thread partials across a 256-thread workgroup; thread t holds part t (valid for t < nparts).
// Returns the total to every thread.
__device__ inline float block_fold(float p, int64_t nparts) {
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

}  // namespace canon
