// attn_i8.hip - the attention kernels of the paper's int8 training path (training-details paragraph on
// int8 computation): the forward P.V product on the int8 matrix cores, quantised per block (R17), and the
// query gradient of the backward accumulated in 64-bit fixed point (R18).
//
// R17.  Blocks are 64 queries x 64 keys of P and 64 keys x head_dim of V.  A block's step is
// RN(amax * RN(1/127)) (amax by bit pattern), its codes come from the R13 quantiser, the product of a P
// block with a V block is an exact int32 sum on v_mfma_i32_32x32x32_i8 (any order: integers), dequantised as
// RN(RN(RN32(acc) * sP) * sV), and O is the R1 sum of these terms over key blocks in ascending order (chains
// of 32 blocks, Algorithm 2 over chains).  Key blocks a query block cannot see are +0 terms and are skipped.
//
// R18.  dQ[i][c] = RN(2^-F * sum over visible keys j of fx(dS[i][j] K[j][c])), fx(p) = the integer nearest to
// p 2^F (ties to even), the sum taken modulo 2^64.  Integer addition modulo 2^64 is associative, so the
// kernel may visit keys in any order.  The fixed-point value of one product is formed without integer
// shifts: for |p 2^F| < 2^51, fma(dS 2^F, K, 1.5 2^52) in binary64 is 1.5 2^52 + rne(p 2^F) exactly (the
// product of two 8-bit significands is exact, and numbers in [2^52, 2^53) are the integers), so the bit
// pattern of that double is a constant plus fx(p); the constants are taken off once at the end.  A key tile
// whose largest |dS| 2^F |K| is not below 2^51 takes an exact path that decomposes the product instead.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

namespace {

constexpr int PVB = 64;                      // R17 block: queries and keys
constexpr uint32_t kInv127Bits = 0x3C010204u;  // RN32(1/127)
constexpr int DQK = 32;                      // R18 keys per staged tile
constexpr double kMagic = 0x1.8p52;          // 1.5 * 2^52
constexpr uint64_t kMagicBits = 0x4338000000000000ull;

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));

// |x| of a bf16 pattern as an ordered integer; a subnormal (read as zero) gives 0
__device__ __forceinline__ uint32_t bf16_mag(uint16_t h) {
  const uint32_t m = h & 0x7FFFu;
  return (m & 0x7F80u) ? m : 0u;
}

__device__ __forceinline__ uint32_t wave_umax(uint32_t v) {
#pragma unroll
  for (int s = 32; s >= 1; s >>= 1) v = max(v, (uint32_t)__shfl_xor((int)v, s, 64));
  return v;
}

// maximum over the workgroup's 256 threads (order-free), returned to every thread
__device__ __forceinline__ uint32_t block_umax(uint32_t v, uint32_t* red) {
  v = wave_umax(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  const uint32_t r = max(max(red[0], red[1]), max(red[2], red[3]));
  __syncthreads();
  return r;
}

// ---- R17 ----------------------------------------------------------------------------------------------

// Codes of one (sequence, key/value head, key block) of V with the block's step.  The codes are written
// transposed, qvt[(bg hd + c) Sp + j], so that each column's keys are contiguous for the matrix operand; keys
// at or beyond S get code 0.
__global__ __launch_bounds__(256) void attn_vquant_kernel(int64_t S, int64_t hd, int64_t Sp,
                                                          const uint16_t* __restrict__ V, int8_t* __restrict__ qvt,
                                                          float* __restrict__ sv) {
  __shared__ uint32_t red[4];
  const int64_t kb = blockIdx.x, bg = blockIdx.y, nb = Sp / PVB;
  const int64_t k0 = kb * PVB;
  const int64_t nk = (S - k0) < PVB ? (S - k0) : PVB;
  const uint16_t* src = V + (bg * S + k0) * hd;
  uint32_t m = 0;
  for (int64_t e = threadIdx.x; e < nk * hd; e += 256) m = max(m, bf16_mag(src[e]));
  m = block_umax(m, red);
  const float step = __uint_as_float(m << 16) * __uint_as_float(kInv127Bits);
  if (threadIdx.x == 0) sv[bg * nb + kb] = step;
  const float st = step_daz(step);
  for (int64_t e = threadIdx.x; e < PVB * hd; e += 256) {
    const int64_t c = e / PVB, j = e % PVB;
    const int8_t q = j < nk ? quant1(bf16_to_f32(src[j * hd + c]), st) : (int8_t)0;
    qvt[(bg * hd + c) * Sp + k0 + j] = q;
  }
}

struct PvArgs {
  const uint16_t* P;  // [B][H][S][S]
  const int8_t* qvt;  // [B][Hkv][hd][Sp]
  const float* sv;    // [B][Hkv][Sp / 64]
  float* of;          // fp32 O, may be null
  uint16_t* ob;       // bf16 O, may be null
  int64_t S, Sp, H, Hkv, hd, window, ldo;
  int vec;  // 16-byte loads of P rows allowed
};

// One workgroup per (sequence, head, query block of 64).  Wavefront w owns rows 32 (w & 1) .. + 31 of the
// block and the 32-column blocks (w >> 1), (w >> 1) + 2, ... of the head dimension (NCB of them).
template <int NCB>
__global__ __launch_bounds__(256) void attn_pv_i8_kernel(PvArgs a) {
  constexpr int LD = PVB + 16;  // padded LDS row (bytes)
  __shared__ __attribute__((aligned(16))) int8_t As[PVB * LD];
  __shared__ __attribute__((aligned(16))) int8_t Bs[64 * NCB * LD];
  __shared__ uint32_t red[4];
  const int64_t S = a.S, W = a.window, hd = a.hd, nb = a.Sp / PVB;
  const int64_t qb = nb - 1 - (int64_t)blockIdx.x;  // longest rows first
  const int64_t bh = blockIdx.y, b = bh / a.H, h = bh % a.H, g = h / (a.H / a.Hkv);
  const int64_t bg = b * a.Hkv + g;
  const int64_t i0 = qb * PVB;
  const uint16_t* Ph = a.P + bh * S * S;
  const int8_t* qv = a.qvt + bg * hd * a.Sp;
  const float* svh = a.sv + bg * nb;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rh = w & 1, cw = w >> 1;
  const int64_t jlo = (W > 0 && i0 - W + 1 > 0) ? i0 - W + 1 : 0;
  const int64_t kb_lo = jlo / PVB, kb_hi = qb;
  // staging: thread t holds P row pr of the block, keys pc .. pc + 15 of the key block
  const int pr = threadIdx.x >> 2, pc = 16 * (threadIdx.x & 3);
  const int64_t pi = i0 + pr;

  float ch[NCB][16], pend[NCB][16], lvl1[NCB][16];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int v = 0; v < 16; ++v) { ch[cb][v] = 0.0f; pend[cb][v] = 0.0f; lvl1[cb][v] = 0.0f; }

  const int64_t c_hi = kb_hi / 32;
  for (int64_t c = 0; c <= c_hi; ++c) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) ch[cb][v] = 0.0f;
    const int64_t kb_a = (32 * c > kb_lo) ? 32 * c : kb_lo;
    const int64_t kb_b = (32 * c + 32 < kb_hi + 1) ? 32 * c + 32 : kb_hi + 1;
    for (int64_t kb = kb_a; kb < kb_b; ++kb) {
      const int64_t k0 = kb * PVB;
      uint16_t pv[16];
      if (a.vec && pi < S && k0 + pc + 16 <= S) {
        const uint4 u0 = *reinterpret_cast<const uint4*>(Ph + pi * S + k0 + pc);
        const uint4 u1 = *reinterpret_cast<const uint4*>(Ph + pi * S + k0 + pc + 8);
        const uint32_t wv[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
#pragma unroll
        for (int e = 0; e < 8; ++e) { pv[2 * e] = (uint16_t)(wv[e] & 0xFFFFu); pv[2 * e + 1] = (uint16_t)(wv[e] >> 16); }
      } else {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int64_t j = k0 + pc + e;
          pv[e] = (pi < S && j < S) ? Ph[pi * S + j] : (uint16_t)0;
        }
      }
      uint32_t m = 0;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int64_t j = k0 + pc + e;
        const bool seen = pi < S && j <= pi && (W == 0 || j > pi - W);
        if (!seen) pv[e] = 0;
        m = max(m, bf16_mag(pv[e]));
      }
      m = block_umax(m, red);
      const float sp = __uint_as_float(m << 16) * __uint_as_float(kInv127Bits);
      const float spd = step_daz(sp);
      uint32_t word[4];
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        uint32_t x = 0;
#pragma unroll
        for (int e = 0; e < 4; ++e) x |= (uint32_t)(uint8_t)quant1(bf16_to_f32(pv[4 * q + e]), spd) << (8 * e);
        word[q] = x;
      }
      *reinterpret_cast<uint4*>(As + pr * LD + pc) = make_uint4(word[0], word[1], word[2], word[3]);
      for (int64_t v = threadIdx.x; v < hd * 4; v += 256) {
        const int64_t col = v >> 2, seg = 16 * (v & 3);
        *reinterpret_cast<uint4*>(Bs + col * LD + seg) = *reinterpret_cast<const uint4*>(qv + col * a.Sp + k0 + seg);
      }
      __syncthreads();
      const float svk = svh[kb];
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        const int colb = cw + 2 * cb;
        if (32 * colb < hd) {
          i32x16 acc;
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[v] = 0;
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) {
            const int kk = 32 * ks + 16 * (lane >> 5);
            const i32x4 av = *reinterpret_cast<const i32x4*>(As + (32 * rh + (lane & 31)) * LD + kk);
            const i32x4 bv = *reinterpret_cast<const i32x4*>(Bs + (32 * colb + (lane & 31)) * LD + kk);
            acc = __builtin_amdgcn_mfma_i32_32x32x32_i8(av, bv, acc, 0, 0, 0);
          }
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const float t = (float)acc[v] * sp;  // RN32 of the integer, then the two dequantising roundings
            const float y = t * svk;
            ch[cb][v] = ch[cb][v] + y;
          }
        }
      }
      __syncthreads();
    }
    // chain c is finished: Algorithm 2 over at most four chain partials
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        if ((c & 1) == 0) {
          pend[cb][v] = ch[cb][v];
        } else {
          const float pair = pend[cb][v] + ch[cb][v];
          lvl1[cb][v] = (c == 1) ? pair : lvl1[cb][v] + pair;
        }
      }
  }
  const int64_t nc = c_hi + 1;  // chains after the last seen block hold +0 and change nothing
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int colb = cw + 2 * cb;
    if (32 * colb >= hd) continue;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      float r = pend[cb][v];
      if (nc == 2 || nc == 4) r = lvl1[cb][v];
      else if (nc == 3) r = lvl1[cb][v] + pend[cb][v];
      const int64_t i = i0 + 32 * rh + (v & 3) + 4 * (lane >> 5) + 8 * (v >> 2);
      const int64_t col = 32 * colb + (lane & 31);
      if (i < S) {
        const int64_t o = (b * S + i) * a.ldo + h * hd + col;
        if (a.of) a.of[o] = r;
        if (a.ob) a.ob[o] = f32_to_bf16(r);
      }
    }
  }
}

// ---- R18 ----------------------------------------------------------------------------------------------

// fx of an exact binary64 product x of two 8-bit significands (any magnitude): nearest integer, ties to
// even, modulo 2^64
__device__ __noinline__ uint64_t fx_exact(double x) {
  if (x == 0.0) return 0;
  const double ax = fabs(x);
  uint64_t u;
  if (ax < 0x1p52) {
    u = (uint64_t)rint(ax);  // rounds half to even; below 2^52, so the conversion is exact
  } else {
    // an integer: significand M (53 bits) times 2^(E - 52); modulo 2^64 the bits shifted past 63 vanish
    const uint64_t bitsx = __double_as_longlong(ax);
    const int64_t E = (int64_t)((bitsx >> 52) & 0x7FF) - 1023;
    const uint64_t M = (bitsx & 0xFFFFFFFFFFFFFull) | (1ull << 52);
    const int64_t sh = E - 52;
    u = sh >= 64 ? 0ull : (M << sh);
  }
  return x < 0.0 ? (uint64_t)0 - u : u;
}

// RN32 of (wrapped sum as int64) * 2^-F under R0: one rounding to 24 bits, then a flush below 2^-126
__device__ float fx_to_f32(uint64_t sum, int F) {
  const int64_t s = (int64_t)sum;
  if (s == 0) return 0.0f;
  const uint32_t sign = s < 0 ? 0x80000000u : 0u;
  const uint64_t u = s < 0 ? (uint64_t)0 - sum : sum;
  const int n = 63 - __builtin_clzll(u);
  uint64_t m;
  int e = n;
  if (n <= 23) {
    m = u << (23 - n);
  } else {
    const int sh = n - 23;
    m = u >> sh;
    const uint64_t rem = u & ((1ull << sh) - 1), half = 1ull << (sh - 1);
    if (rem > half || (rem == half && (m & 1))) ++m;
    if (m == (1ull << 24)) { m >>= 1; ++e; }
  }
  const int be = e - F + 127;
  if (be < 1) return __uint_as_float(sign);
  return __uint_as_float(sign | ((uint32_t)be << 23) | ((uint32_t)m & 0x7FFFFFu));
}

struct DqArgs {
  const uint16_t* dS;  // [B][H][S][S]
  const uint16_t* K;   // [B][Hkv][S][hd]
  float* dQ;           // [B][S][ldq], head h at columns h hd ..
  int64_t S, H, Hkv, hd, window, ldq;
  int F;
  int vec;  // 16-byte loads of dS rows allowed
};

// One workgroup per (sequence, head, query block of 64); thread t accumulates rows 4 (t / 16) .. + 3 and
// columns C (t % 16) .. + C - 1 (hd = 16 C) in 64-bit integers.
template <int C>
__global__ __launch_bounds__(256) void attn_dq_fixed_kernel(DqArgs a) {
  constexpr int HD = 16 * C;
  __shared__ __attribute__((aligned(16))) double ds_t[DQK][64];  // [key][row]: dS 2^F, masked entries 0
  __shared__ __attribute__((aligned(16))) double k_t[DQK][HD];   // [key][column]: K
  __shared__ uint32_t red[4];
  const int64_t S = a.S, W = a.window;
  const int64_t nqb = (S + 63) / 64;
  const int64_t qb = nqb - 1 - (int64_t)blockIdx.x;  // longest rows first
  const int64_t bh = blockIdx.y, b = bh / a.H, h = bh % a.H, g = h / (a.H / a.Hkv);
  const int64_t i0 = qb * 64, i1 = (i0 + 64 < S) ? i0 + 64 : S;
  const uint16_t* dSh = a.dS + bh * S * S;
  const uint16_t* Kh = a.K + (b * a.Hkv + g) * S * HD;
  const int rg = threadIdx.x >> 4, cg = threadIdx.x & 15;
  const double two_f = ldexp(1.0, a.F);
  uint64_t acc[4][C];
#pragma unroll
  for (int r = 0; r < 4; ++r)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[r][c] = 0;
  const int64_t jlo = (W > 0 && i0 - W + 1 > 0) ? i0 - W + 1 : 0;
  const int64_t t_lo = jlo / DQK, t_hi = (i1 - 1) / DQK;
  uint64_t n_fast = 0;  // keys added through the fast path (each added kMagicBits once per output)
  const int sr = threadIdx.x >> 2, sk = 8 * (threadIdx.x & 3);  // dS staging: row sr, keys sk .. sk + 7
  const int64_t si = i0 + sr;
  for (int64_t kt = t_lo; kt <= t_hi; ++kt) {
    const int64_t j0 = kt * DQK;
    uint32_t dmag = 0, kmag = 0;
    {
      uint16_t v[8];
      if (a.vec && si < S && j0 + sk + 8 <= S) {
        const uint4 u = *reinterpret_cast<const uint4*>(dSh + si * S + j0 + sk);
        const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) { v[2 * e] = (uint16_t)(wv[e] & 0xFFFFu); v[2 * e + 1] = (uint16_t)(wv[e] >> 16); }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const int64_t j = j0 + sk + e;
          v[e] = (si < S && j < S) ? dSh[si * S + j] : (uint16_t)0;
        }
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t j = j0 + sk + e;
        const bool seen = si < S && j <= si && (W == 0 || j > si - W);
        const uint16_t x = seen ? v[e] : (uint16_t)0;
        dmag = max(dmag, bf16_mag(x));
        ds_t[sk + e][sr] = (double)bf16_to_f32(x) * two_f;
      }
    }
    for (int e = threadIdx.x; e < DQK * HD; e += 256) {
      const int kk = e / HD, col = e % HD;
      const int64_t j = j0 + kk;
      const uint16_t x = j < S ? Kh[j * HD + col] : (uint16_t)0;
      kmag = max(kmag, bf16_mag(x));
      k_t[kk][col] = (double)bf16_to_f32(x);
    }
    dmag = block_umax(dmag, red);  // its barriers also publish the staged tiles
    kmag = block_umax(kmag, red);
    const double bound = (double)__uint_as_float(dmag << 16) * two_f * (double)__uint_as_float(kmag << 16);
    if (bound < 0x1p51) {
      n_fast += DQK;
#pragma unroll 4
      for (int kk = 0; kk < DQK; ++kk) {
        double dv[4], kv[C];
#pragma unroll
        for (int r = 0; r < 4; ++r) dv[r] = ds_t[kk][4 * rg + r];
#pragma unroll
        for (int c = 0; c < C; ++c) kv[c] = k_t[kk][C * cg + c];
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int c = 0; c < C; ++c) acc[r][c] += (uint64_t)__double_as_longlong(__builtin_fma(dv[r], kv[c], kMagic));
      }
    } else {
      for (int kk = 0; kk < DQK; ++kk)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int c = 0; c < C; ++c) acc[r][c] += fx_exact(ds_t[kk][4 * rg + r] * k_t[kk][C * cg + c]);
    }
    __syncthreads();
  }
  const uint64_t bias = n_fast * kMagicBits;
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int64_t i = i0 + 4 * rg + r;
    if (i >= S) continue;
#pragma unroll
    for (int c = 0; c < C; ++c)
      a.dQ[(b * S + i) * a.ldq + h * HD + C * cg + c] = fx_to_f32(acc[r][c] - bias, a.F);
  }
}

}  // namespace

int64_t attn_pv_blocks(int64_t S) { return (S + PVB - 1) / PVB; }

hipError_t attn_pv_i8_launch(int64_t B, int64_t H, int64_t Hkv, int64_t S, int64_t hd, int64_t window,
                             const uint16_t* P, const uint16_t* V, float* of, uint16_t* ob, int64_t ldo, int8_t* qvt,
                             float* sv, hipStream_t s) {
  if (B == 0) return hipSuccess;
  const int64_t nb = attn_pv_blocks(S), Sp = nb * PVB;
  hipLaunchKernelGGL(attn_vquant_kernel, dim3((unsigned)nb, (unsigned)(B * Hkv)), dim3(256), 0, s, S, hd, Sp, V, qvt,
                     sv);
  PvArgs a;
  a.P = P; a.qvt = qvt; a.sv = sv; a.of = of; a.ob = ob;
  a.S = S; a.Sp = Sp; a.H = H; a.Hkv = Hkv; a.hd = hd; a.window = window; a.ldo = ldo;
  a.vec = (S % 8 == 0) && (((uintptr_t)P & 15) == 0);
  const dim3 grid((unsigned)nb, (unsigned)(B * H));
  if (hd <= 64) hipLaunchKernelGGL(attn_pv_i8_kernel<1>, grid, dim3(256), 0, s, a);
  else if (hd <= 128) hipLaunchKernelGGL(attn_pv_i8_kernel<2>, grid, dim3(256), 0, s, a);
  else hipLaunchKernelGGL(attn_pv_i8_kernel<4>, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t attn_dq_fixed_launch(int64_t B, int64_t H, int64_t Hkv, int64_t S, int64_t hd, int64_t window, int F,
                                const uint16_t* dS, const uint16_t* K, float* dQ, int64_t ldq, hipStream_t s) {
  if (B == 0) return hipSuccess;
  DqArgs a;
  a.dS = dS; a.K = K; a.dQ = dQ;
  a.S = S; a.H = H; a.Hkv = Hkv; a.hd = hd; a.window = window; a.ldq = ldq; a.F = F;
  a.vec = (S % 8 == 0) && (((uintptr_t)dS & 15) == 0);
  const dim3 grid((unsigned)((S + 63) / 64), (unsigned)(B * H));
  switch (hd) {
    case 16: hipLaunchKernelGGL(attn_dq_fixed_kernel<1>, grid, dim3(256), 0, s, a); break;
    case 32: hipLaunchKernelGGL(attn_dq_fixed_kernel<2>, grid, dim3(256), 0, s, a); break;
    case 64: hipLaunchKernelGGL(attn_dq_fixed_kernel<4>, grid, dim3(256), 0, s, a); break;
    case 128: hipLaunchKernelGGL(attn_dq_fixed_kernel<8>, grid, dim3(256), 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace canon
