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
// whose largest |dS| 2^F |K| is not below 2^51 takes a longer exact form for its products (fx_any).
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

namespace {

constexpr int PVB = 64;                      // R17 block: queries and keys
constexpr uint32_t kInv127Bits = 0x3C010204u;  // RN32(1/127)
constexpr int DQK = 16;                      // R18 keys per staged tile
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
  const bool recip = recip_step_ok(st);
  const float rst = recip ? 1.0f / st : 0.0f;
  for (int64_t e = threadIdx.x; e < PVB * hd; e += 256) {
    const int64_t c = e / PVB, j = e % PVB;
    const float vf = j < nk ? bf16_to_f32(src[j * hd + c]) : 0.0f;
    const int8_t q = j < nk ? (recip ? quant_recip(vf, st, rst) : quant1(vf, st)) : (int8_t)0;
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
// block and the 32-column blocks (w >> 1), (w >> 1) + 2, ... of the head dimension (NCB of them).  Per key
// block: the P tile (already in registers) is masked and its absmax reduced (shuffles, then four wavefront
// maxima through LDS); the codes of P and of V go to LDS, while later key blocks' P tiles and V codes load
// into registers and the matrix instructions and the dequantising chain run.  LDS tiles and the maxima
// are double buffered, so each key block takes two barriers; the operands of the next three key blocks are
// in flight in registers.
template <int NCB>
__global__ __launch_bounds__(256) void attn_pv_i8_kernel(PvArgs a) {
  constexpr int LD = PVB + 16;  // padded LDS row (bytes)
  constexpr int NVQ = NCB;      // 16-byte V-code vectors per thread (hd * 4 vectors of a block / 256 threads)
  __shared__ __attribute__((aligned(16))) int8_t As[2][PVB * LD];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][64 * NCB * LD];
  __shared__ uint32_t red[2][4];
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

  // 16 bf16 values as 8 words (element e in the low or high half of word e / 2)
  auto load_p = [&](int64_t kb, uint32_t (&pw)[8]) __attribute__((always_inline)) {
    const int64_t k0 = kb * PVB;
    if (a.vec && pi < S && k0 + pc + 16 <= S) {
      const uint4 u0 = *reinterpret_cast<const uint4*>(Ph + pi * S + k0 + pc);
      const uint4 u1 = *reinterpret_cast<const uint4*>(Ph + pi * S + k0 + pc + 8);
      pw[0] = u0.x; pw[1] = u0.y; pw[2] = u0.z; pw[3] = u0.w;
      pw[4] = u1.x; pw[5] = u1.y; pw[6] = u1.z; pw[7] = u1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int64_t j = k0 + pc + 2 * e;
        const uint32_t lo = (pi < S && j < S) ? Ph[pi * S + j] : 0u;
        const uint32_t hi = (pi < S && j + 1 < S) ? Ph[pi * S + j + 1] : 0u;
        pw[e] = lo | (hi << 16);
      }
    }
  };
  auto load_v = [&](int64_t kb, uint32_t (&vq)[4 * NVQ]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < NVQ; ++q) {
      const int64_t v = threadIdx.x + 256 * q;
      if (v < hd * 4) {
        const uint4 u = *reinterpret_cast<const uint4*>(qv + (v >> 2) * a.Sp + kb * PVB + 16 * (v & 3));
        vq[4 * q] = u.x; vq[4 * q + 1] = u.y; vq[4 * q + 2] = u.z; vq[4 * q + 3] = u.w;
      }
    }
  };

  float ch[NCB][16], pend[NCB][16], lvl1[NCB][16];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
    for (int v = 0; v < 16; ++v) { ch[cb][v] = 0.0f; pend[cb][v] = 0.0f; lvl1[cb][v] = 0.0f; }
  // chain c of the R1 sum over key blocks is finished: Algorithm 2 over at most four chain partials (uniform
  // branches with whole-array loops, so the arrays stay in registers)
  auto finish_chain = [&](int64_t c) __attribute__((always_inline)) {
    if ((c & 1) == 0) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int v = 0; v < 16; ++v) pend[cb][v] = ch[cb][v];
    } else if (c == 1) {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int v = 0; v < 16; ++v) lvl1[cb][v] = pend[cb][v] + ch[cb][v];
    } else {
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
        for (int v = 0; v < 16; ++v) lvl1[cb][v] = lvl1[cb][v] + (pend[cb][v] + ch[cb][v]);
    }
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) ch[cb][v] = 0.0f;
  };

  // chains wholly before the first visible block hold +0: with pend = lvl1 = +0 the fold state is already
  // what finishing them would leave
  int64_t cur_c = kb_lo / 32;
  // one key block: its operands (pws, vqs, svs) were loaded three blocks earlier; once staged, the same
  // registers receive the operands of block kb + 3
  auto step = [&](int64_t kb, int buf, uint32_t (&pws)[8], uint32_t (&vqs)[4 * NVQ], float& svs)
                  __attribute__((always_inline)) {
    if ((kb & 31) == 0 && kb != kb_lo) {  // the previous block closed chain cur_c
      finish_chain(cur_c);
      ++cur_c;
    }
    const int64_t k0 = kb * PVB;
    uint32_t pwv[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) pwv[e] = pws[e];
    uint32_t m = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int64_t j = k0 + pc + e;
      const bool seen = pi < S && j <= pi && (W == 0 || j > pi - W);
      const uint32_t keep = seen ? (0xFFFFu << (16 * (e & 1))) : 0u;
      pwv[e >> 1] &= keep | (0xFFFFu << (16 * ((e & 1) ^ 1)));
      m = max(m, bf16_mag((uint16_t)(pwv[e >> 1] >> (16 * (e & 1)))));
    }
    m = wave_umax(m);
    if (lane == 0) red[buf][w] = m;
    __syncthreads();
    m = max(max(red[buf][0], red[buf][1]), max(red[buf][2], red[buf][3]));
    const float sp = __uint_as_float(m << 16) * __uint_as_float(kInv127Bits);
    const float spd = step_daz(sp);
    const bool recip = recip_step_ok(spd);
    const float rsp = recip ? 1.0f / spd : 0.0f;
    uint32_t word0 = 0, word1 = 0, word2 = 0, word3 = 0;
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const float pf = bf16_to_f32((uint16_t)(pwv[e >> 1] >> (16 * (e & 1))));
      const int8_t c = recip ? quant_recip(pf, spd, rsp) : quant1(pf, spd);
      const uint32_t bits = (uint32_t)(uint8_t)c << (8 * (e & 3));
      if (e < 4) word0 |= bits;
      else if (e < 8) word1 |= bits;
      else if (e < 12) word2 |= bits;
      else word3 |= bits;
    }
    *reinterpret_cast<uint4*>(As[buf] + pr * LD + pc) = make_uint4(word0, word1, word2, word3);
#pragma unroll
    for (int q = 0; q < NVQ; ++q) {
      const int64_t v = threadIdx.x + 256 * q;
      if (v < hd * 4)
        *reinterpret_cast<uint4*>(Bs[buf] + (v >> 2) * LD + 16 * (v & 3)) =
            make_uint4(vqs[4 * q], vqs[4 * q + 1], vqs[4 * q + 2], vqs[4 * q + 3]);
    }
    const float svk = svs;
    if (kb + 3 <= kb_hi) {
      load_p(kb + 3, pws);
      load_v(kb + 3, vqs);
      svs = svh[kb + 3];
    }
    __syncthreads();
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
          const i32x4 av = *reinterpret_cast<const i32x4*>(As[buf] + (32 * rh + (lane & 31)) * LD + kk);
          const i32x4 bv = *reinterpret_cast<const i32x4*>(Bs[buf] + (32 * colb + (lane & 31)) * LD + kk);
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
  };

  uint32_t pa[8], pb[8], pcx[8];
  uint32_t va[4 * NVQ], vb[4 * NVQ], vc[4 * NVQ];
  float sa = 0.0f, sb = 0.0f, sc = 0.0f;
  load_p(kb_lo, pa); load_v(kb_lo, va); sa = svh[kb_lo];
  if (kb_lo + 1 <= kb_hi) { load_p(kb_lo + 1, pb); load_v(kb_lo + 1, vb); sb = svh[kb_lo + 1]; }
  if (kb_lo + 2 <= kb_hi) { load_p(kb_lo + 2, pcx); load_v(kb_lo + 2, vc); sc = svh[kb_lo + 2]; }
  for (int64_t kb = kb_lo; kb <= kb_hi; kb += 3) {
    step(kb, 0, pa, va, sa);
    if (kb + 1 <= kb_hi) step(kb + 1, 1, pb, vb, sb);
    if (kb + 2 <= kb_hi) step(kb + 2, 0, pcx, vc, sc);
  }
  finish_chain(cur_c);
  const int64_t nc = cur_c + 1;  // chains after the last seen block hold +0 and change nothing
  // the fold's result: one chain, pend; two or four, lvl1; three, lvl1 + pend (into ch)
  if (nc == 1) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) ch[cb][v] = pend[cb][v];
  } else if (nc == 3) {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) ch[cb][v] = lvl1[cb][v] + pend[cb][v];
  } else {
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int v = 0; v < 16; ++v) ch[cb][v] = lvl1[cb][v];
  }
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) {
    const int colb = cw + 2 * cb;
    if (32 * colb >= hd) continue;
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int64_t i = i0 + 32 * rh + (v & 3) + 4 * (lane >> 5) + 8 * (v >> 2);
      const int64_t col = 32 * colb + (lane & 31);
      if (i < S) {
        const int64_t o = (b * S + i) * a.ldo + h * hd + col;
        if (a.of) a.of[o] = ch[cb][v];
        if (a.ob) a.ob[o] = f32_to_bf16(ch[cb][v]);
      }
    }
  }
}

// ---- R18 ----------------------------------------------------------------------------------------------

// fx of an exact binary64 product x of two 8-bit significands, any magnitude, without branches.  Below 2^51
// the magic-number rounding applies.  Otherwise x = m 2^e with m < 2^16 and e >= 35 is an integer divisible
// by 2^35, and fx(x) = x modulo 2^64: |x| minus its multiple of 2^64 is exact (a multiple of 2^35 below
// 2^64), and is hi 2^32 with hi < 2^32 an exact unsigned conversion; the sign is applied modulo 2^64.
__device__ __forceinline__ uint64_t fx_any(double x) {
  const double ax = fabs(x);
  const uint64_t small = (uint64_t)__double_as_longlong(__builtin_fma(x, 1.0, kMagic)) - kMagicBits;
  const double q = trunc(ax * 0x1p-64);
  const double r = __builtin_fma(-q, 0x1p64, ax);
  const uint32_t hi = (uint32_t)(r * 0x1p-32);
  uint64_t big = (uint64_t)hi << 32;
  big = x < 0.0 ? (uint64_t)0 - big : big;
  return ax < 0x1p51 ? small : big;
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
  int64_t B, S, H, Hkv, hd, window, ldq;
  int F;
  int vec;  // 16-byte loads of dS and K rows allowed
};

constexpr int DQB = 128;  // R18 query rows per workgroup

// Workgroup -> (query block, sequence x head): the query block index is the slow one and descends, so the
// whole launch runs its longest rows first (with heads as the fast index, the long blocks of the last heads
// would start late and leave a tail).
__device__ __forceinline__ void dq_block(const DqArgs& a, int64_t& qb, int64_t& bh) {
  const int64_t nbh = a.B * a.H, nqb = (a.S + DQB - 1) / DQB;
  qb = nqb - 1 - (int64_t)blockIdx.x / nbh;
  bh = (int64_t)blockIdx.x % nbh;
}

// The key tiles of one query block, summed into acc.  EXACT = false: the magic-number form (fast); a tile
// whose bound |dS| 2^F |K| reaches 2^51 makes the call return true, and the caller runs the tiles again with
// EXACT = true (fx_any for every product).  Key tiles of 16: the staged tile is converted to binary64 in
// LDS (dS times 2^F, masked entries 0) while the next tile's bf16 values are loaded into registers; two
// barriers per tile.
template <int C, bool EXACT>
__device__ __forceinline__ bool dq_tiles(const DqArgs& a, double (*ds_t)[DQB], double (*k_t)[16 * C],
                                         uint32_t (*red)[2][4], uint64_t (&acc)[8][C], uint64_t& n_fast) {
  constexpr int HD = 16 * C;
  constexpr int KV = (DQK * HD / 8 + 255) / 256;  // 16-byte K vectors per thread per tile
  const int64_t S = a.S, W = a.window;
  int64_t qb, bh;
  dq_block(a, qb, bh);
  const int64_t b = bh / a.H, h = bh % a.H, g = h / (a.H / a.Hkv);
  const int64_t i0 = qb * DQB, i1 = (i0 + DQB < S) ? i0 + DQB : S;
  const uint16_t* dSh = a.dS + bh * S * S;
  const uint16_t* Kh = a.K + (b * a.Hkv + g) * S * HD;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int rg = threadIdx.x >> 4, cg = threadIdx.x & 15;
  const double two_f = ldexp(1.0, a.F);
  const int64_t jlo = (W > 0 && i0 - W + 1 > 0) ? i0 - W + 1 : 0;
  const int64_t t_lo = jlo / DQK, t_hi = (i1 - 1) / DQK;
  const int sr = threadIdx.x >> 1, sk = 8 * (threadIdx.x & 1);  // dS staging: row sr, keys sk .. sk + 7
  const int64_t si = i0 + sr;
  bool slow = false;

  auto load_ds = [&](int64_t kt, uint16_t (&v)[8]) __attribute__((always_inline)) {
    const int64_t j0 = kt * DQK;
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
  };
  auto load_k = [&](int64_t kt, uint16_t (&v)[KV][8]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < KV; ++q) {
      const int e = threadIdx.x + 256 * q;  // vector e: key e / (HD / 8), columns 8 (e % (HD / 8)) ..
      const int kk = e / (HD / 8), c0 = 8 * (e % (HD / 8));
      const int64_t j = kt * DQK + kk;
      if (kk < DQK && j < S) {
        if (a.vec) {
          const uint4 u = *reinterpret_cast<const uint4*>(Kh + j * HD + c0);
          const uint32_t wv[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
          for (int x = 0; x < 4; ++x) { v[q][2 * x] = (uint16_t)(wv[x] & 0xFFFFu); v[q][2 * x + 1] = (uint16_t)(wv[x] >> 16); }
        } else {
#pragma unroll
          for (int x = 0; x < 8; ++x) v[q][x] = Kh[j * HD + c0 + x];
        }
      } else {
#pragma unroll
        for (int x = 0; x < 8; ++x) v[q][x] = 0;
      }
    }
  };

  uint16_t dv16[8], kv16[KV][8];
  load_ds(t_lo, dv16);
  load_k(t_lo, kv16);
  int buf = 0;
  for (int64_t kt = t_lo; kt <= t_hi; ++kt, buf ^= 1) {
    const int64_t j0 = kt * DQK;
    uint32_t dmag = 0, kmag = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int64_t j = j0 + sk + e;
      const bool seen = si < S && j <= si && (W == 0 || j > si - W);
      const uint16_t x = seen ? dv16[e] : (uint16_t)0;
      dmag = max(dmag, bf16_mag(x));
      ds_t[sk + e][sr] = (double)bf16_to_f32(x) * two_f;
    }
#pragma unroll
    for (int q = 0; q < KV; ++q) {
      const int e = threadIdx.x + 256 * q;
      const int kk = e / (HD / 8), c0 = 8 * (e % (HD / 8));
      if (kk < DQK) {
#pragma unroll
        for (int x = 0; x < 8; ++x) {
          kmag = max(kmag, bf16_mag(kv16[q][x]));
          k_t[kk][c0 + x] = (double)bf16_to_f32(kv16[q][x]);
        }
      }
    }
    if (!EXACT) {
      dmag = wave_umax(dmag);
      kmag = wave_umax(kmag);
      if (lane == 0) { red[buf][0][w] = dmag; red[buf][1][w] = kmag; }
    }
    __syncthreads();
    if (kt < t_hi) {  // the next tile travels while this one is multiplied
      load_ds(kt + 1, dv16);
      load_k(kt + 1, kv16);
    }
    if (!EXACT) {
      dmag = max(max(red[buf][0][0], red[buf][0][1]), max(red[buf][0][2], red[buf][0][3]));
      kmag = max(max(red[buf][1][0], red[buf][1][1]), max(red[buf][1][2], red[buf][1][3]));
      const double bound = (double)__uint_as_float(dmag << 16) * two_f * (double)__uint_as_float(kmag << 16);
      slow |= !(bound < 0x1p51);
      n_fast += DQK;
#pragma unroll 1
      for (int kk = 0; kk < DQK; ++kk) {
        double dv[8], kv[C];
#pragma unroll
        for (int r = 0; r < 8; ++r) dv[r] = ds_t[kk][8 * rg + r];
#pragma unroll
        for (int c = 0; c < C; ++c) kv[c] = k_t[kk][C * cg + c];
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
          for (int c = 0; c < C; ++c) acc[r][c] += (uint64_t)__double_as_longlong(__builtin_fma(dv[r], kv[c], kMagic));
      }
    } else {
#pragma unroll 1
      for (int kk = 0; kk < DQK; ++kk) {
        double dv[8], kv[C];
#pragma unroll
        for (int r = 0; r < 8; ++r) dv[r] = ds_t[kk][8 * rg + r];
#pragma unroll
        for (int c = 0; c < C; ++c) kv[c] = k_t[kk][C * cg + c];
#pragma unroll
        for (int r = 0; r < 8; ++r)
#pragma unroll
          for (int c = 0; c < C; ++c) acc[r][c] += fx_any(dv[r] * kv[c]);
      }
    }
    __syncthreads();
  }
  return slow;
}

// One workgroup per (sequence, head, query block of 128); thread t accumulates rows 8 (t / 16) .. + 7 and
// columns C (t % 16) .. + C - 1 (hd = 16 C) in 64-bit integers.
template <int C>
__global__ __launch_bounds__(256) void attn_dq_fixed_kernel(DqArgs a) {
  constexpr int HD = 16 * C;
  __shared__ __attribute__((aligned(16))) double ds_t[DQK][DQB];  // [key][row]
  __shared__ __attribute__((aligned(16))) double k_t[DQK][HD];    // [key][column]
  __shared__ uint32_t red[2][2][4];
  uint64_t acc[8][C];
#pragma unroll
  for (int r = 0; r < 8; ++r)
#pragma unroll
    for (int c = 0; c < C; ++c) acc[r][c] = 0;
  uint64_t n_fast = 0;  // keys added through the fast form (each added kMagicBits once per output)
  if (dq_tiles<C, false>(a, ds_t, k_t, red, acc, n_fast)) {  // uniform over the workgroup
#pragma unroll
    for (int r = 0; r < 8; ++r)
#pragma unroll
      for (int c = 0; c < C; ++c) acc[r][c] = 0;
    n_fast = 0;
    dq_tiles<C, true>(a, ds_t, k_t, red, acc, n_fast);
  }
  const int64_t S = a.S;
  int64_t qb, bh;
  dq_block(a, qb, bh);
  const int64_t b = bh / a.H, h = bh % a.H;
  const int rg = threadIdx.x >> 4, cg = threadIdx.x & 15;
  const uint64_t bias = n_fast * kMagicBits;
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int64_t i = qb * DQB + 8 * rg + r;
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
  a.B = B; a.S = S; a.H = H; a.Hkv = Hkv; a.hd = hd; a.window = window; a.ldq = ldq; a.F = F;
  a.vec = (S % 8 == 0) && (((uintptr_t)dS & 15) == 0) && (((uintptr_t)K & 15) == 0);
  const int64_t nwg = (S + DQB - 1) / DQB * B * H;
  if (nwg == 0) return hipSuccess;
  if (nwg > 0xFFFFFFFFll) return hipErrorInvalidValue;
  const dim3 grid((unsigned)nwg);
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
