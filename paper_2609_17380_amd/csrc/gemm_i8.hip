// gemm_i8.hip - exact int8 GEMM on the int8 matrix cores, with the dequantisation epilogue of the int8
// quantised linear.
//
// acc[i][j] = sum over k of a[i][k] * b[j][k] with int8 operands (a [m][k], b [n][k], both k-contiguous,
// b holding one output column per row as weights [out][in] do).  Integer products and sums are exact, and
// |acc| < 2^31 for k <= 65536, so every summation order gives the same int32: the k loop may be split,
// reordered and spread over matrix instructions freely.  The dequantised output is
// y[i][j] = RN(RN(RN32(acc) * sa) * sb[j]).
//
// Tiling: whole 256 x 256 tiles (m, n multiples of 256) run on 4 wavefronts, each a 128 x 128 block of
// 4 x 4 v_mfma_i32_32x32x32_i8 instructions (gemm_i8_tile_kernel).  Other shapes: a workgroup of NW wavefronts
// owns a 16 NW HB x 64 WN output tile, each wavefront a 32 HB x 32 WN block: 256 x 256 tiles of 8 wavefronts
// with 64-byte stages for large products, else 128 x 128 tiles of 4 wavefronts with 128-byte stages.  Stages of KS k bytes are staged
// through LDS (rows padded by 16 bytes, which keeps the 16-byte operand reads of 32 consecutive rows free of
// bank conflicts), double buffered.
// Each lane of a 32x32x32 instruction supplies 16 consecutive k bytes of one row of A and of B; the two
// half-wavefronts cover k 0..15 and 16..31 of the instruction's 32.
#include <hip/hip_runtime.h>

#include "canon_internal.h"

namespace canon {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));

// Workgroup configuration: NW wavefronts in (NW / 2) x 2, wavefront (wr, wc) owning rows [32 HB wr, 32 HB (wr + 1))
// and columns [32 WN wc, 32 WN (wc + 1)) of a BM x (64 WN) tile (HB x WN instruction blocks); stages of KS k bytes.
template <int HB, int WN, int KS, int NW>
struct I8Cfg {
  static constexpr int BM = 16 * NW * HB;     // workgroup tile rows
  static constexpr int NT = 64 * NW;          // threads
  static constexpr int BN = 64 * WN;          // workgroup tile columns
  static constexpr int LD = KS + 16;          // padded LDS row (bytes)
  static constexpr int AV = BM * KS / 16 / NT;  // 16-byte vectors of A per thread per stage
  static constexpr int BV = BN * KS / 16 / NT;  // ... of B
  static_assert(AV * NT * 16 == BM * KS && BV * NT * 16 == BN * KS, "whole vectors per thread");
};

template <class Cf>
struct I8Raw {
  uint4 a[Cf::AV], b[Cf::BV];
};

// 16 consecutive bytes of which the first `valid` exist (zero fill beyond)
template <bool FAST>
__device__ __forceinline__ uint4 ld16(const int8_t* p, int64_t valid, bool vec) {
  if (FAST || (vec && valid >= 16)) return *reinterpret_cast<const uint4*>(p);
  uint32_t w[4] = {0u, 0u, 0u, 0u};
  for (int e = 0; e < 16; ++e)
    if (e < valid) w[e >> 2] |= (uint32_t)(uint8_t)p[e] << (8 * (e & 3));
  return make_uint4(w[0], w[1], w[2], w[3]);
}

// Global -> registers for the stage starting at k0: vector idx = t + NT it covers row idx / (KS/16),
// 16-byte segment idx % (KS/16) of the row's KS bytes.
template <class Cf, int KS, bool FAST>
__device__ __forceinline__ I8Raw<Cf> load_stage(const GemmI8Args& g, int64_t row0, int64_t col0, int64_t k0) {
  constexpr int SEG = KS / 16;
  const int t = threadIdx.x;
  I8Raw<Cf> r;
#pragma unroll
  for (int it = 0; it < Cf::AV; ++it) {
    const int idx = t + Cf::NT * it;
    const int64_t k = k0 + 16 * (idx % SEG), row = row0 + idx / SEG;
    r.a[it] = ld16<FAST>(g.a + row * g.lda + k, (row < g.m) ? g.k - k : 0, g.vec);
  }
#pragma unroll
  for (int it = 0; it < Cf::BV; ++it) {
    const int idx = t + Cf::NT * it;
    const int64_t k = k0 + 16 * (idx % SEG), col = col0 + idx / SEG;
    r.b[it] = ld16<FAST>(g.b + col * g.ldb + k, (col < g.n) ? g.k - k : 0, g.vec);
  }
  return r;
}

template <class Cf, int KS>
__device__ __forceinline__ void store_stage(int8_t* As, int8_t* Bs, const I8Raw<Cf>& r) {
  constexpr int SEG = KS / 16;
  const int t = threadIdx.x;
#pragma unroll
  for (int it = 0; it < Cf::AV; ++it) {
    const int idx = t + Cf::NT * it;
    *reinterpret_cast<uint4*>(As + (idx / SEG) * Cf::LD + 16 * (idx % SEG)) = r.a[it];
  }
#pragma unroll
  for (int it = 0; it < Cf::BV; ++it) {
    const int idx = t + Cf::NT * it;
    *reinterpret_cast<uint4*>(Bs + (idx / SEG) * Cf::LD + 16 * (idx % SEG)) = r.b[it];
  }
}

template <int HB, int WN, int KS, int NW>
__global__ __launch_bounds__(64 * NW) void gemm_i8_kernel(GemmI8Args g) {
  using Cf = I8Cfg<HB, WN, KS, NW>;
  constexpr int BM = Cf::BM, BN = Cf::BN, LD = Cf::LD;
  __shared__ __attribute__((aligned(16))) int8_t As[2][BM * LD];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][BN * LD];

  // tile order: a contiguous run of tiles per XCD, walked in groups of 8 tile rows
  constexpr int64_t GM = 8;
  const int64_t tiles_n = (g.n + BN - 1) / BN;
  const int64_t tiles_m = (g.m + BM - 1) / BM;
  const int64_t tiles = tiles_m * tiles_n;
  int64_t tile = blockIdx.x;
  if ((tiles & 7) == 0) tile = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int64_t group = tile / (GM * tiles_n);
  const int64_t first_m = group * GM;
  const int64_t gsize = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
  const int64_t within = tile - group * GM * tiles_n;
  const int64_t row0 = (first_m + within % gsize) * BM, col0 = (within / gsize) * BN;
  const bool tile_in = g.vec && row0 + BM <= g.m && col0 + BN <= g.n;

  // wavefront (wr, wc) owns rows [32 HB wr, 32 HB (wr + 1)) and columns [32 WN wc, 32 WN (wc + 1)) of the tile
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int ar = 32 * HB * wr + (lane & 31), bc = 32 * WN * wc + (lane & 31);
  const int kh = 16 * (lane >> 5);

  i32x16 acc[HB][WN];
#pragma unroll
  for (int h = 0; h < HB; ++h)
#pragma unroll
    for (int v2 = 0; v2 < WN; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[h][v2][v] = 0;

  const int64_t ns = (g.k + KS - 1) / KS;
  int buf = 0;
  if (ns > 0) store_stage<Cf, KS>(As[0], Bs[0], load_stage<Cf, KS, false>(g, row0, col0, 0));
  __syncthreads();
  for (int64_t s = 0; s < ns; ++s) {
    const bool more = s + 1 < ns;
    I8Raw<Cf> nxt;
    if (more) {
      if (tile_in && (s + 2) * KS <= g.k) nxt = load_stage<Cf, KS, true>(g, row0, col0, (s + 1) * KS);
      else nxt = load_stage<Cf, KS, false>(g, row0, col0, (s + 1) * KS);
    }
    __builtin_amdgcn_sched_barrier(0);
    const int8_t* as = As[buf];
    const int8_t* bs = Bs[buf];
#pragma unroll
    for (int ks = 0; ks < KS / 32; ++ks) {
      const int kk = 32 * ks + kh;
      i32x4 a[HB], b[WN];
#pragma unroll
      for (int h = 0; h < HB; ++h) a[h] = *reinterpret_cast<const i32x4*>(as + (ar + 32 * h) * LD + kk);
#pragma unroll
      for (int v2 = 0; v2 < WN; ++v2) b[v2] = *reinterpret_cast<const i32x4*>(bs + (bc + 32 * v2) * LD + kk);
#pragma unroll
      for (int h = 0; h < HB; ++h)
#pragma unroll
        for (int v2 = 0; v2 < WN; ++v2)
          acc[h][v2] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[h], b[v2], acc[h][v2], 0, 0, 0);
    }
    __builtin_amdgcn_sched_barrier(0);
    if (more) store_stage<Cf, KS>(As[buf ^ 1], Bs[buf ^ 1], nxt);
    __syncthreads();
    buf ^= 1;
  }

  // result layout: register v, lane l -> row (v % 4) + 4 (l / 32) + 8 (v / 4), column l % 32 of the block
  const float sa = g.y ? *g.sa : 0.0f;
#pragma unroll
  for (int h = 0; h < HB; ++h)
#pragma unroll
    for (int v2 = 0; v2 < WN; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int64_t i = row0 + 32 * HB * wr + 32 * h + (v & 3) + 4 * (lane >> 5) + 8 * (v >> 2);
        const int64_t j = col0 + 32 * WN * wc + 32 * v2 + (lane & 31);
        if (i < g.m && j < g.n) {
          const int32_t a = acc[h][v2][v];
          if (g.acc) g.acc[i * g.ldc + j] = a;
          if (g.y) {
            const float af = (float)a;  // round to nearest even
            const float t = af * sa;
            g.y[i * g.ldc + j] = t * g.sb[g.sb_scalar ? 0 : j];
          }
        }
      }
}

// Whole 256 x 256 tiles (m, n multiples of 256, k of KS, 16-byte aligned rows): 4 wavefronts, each a 128 x 128
// block of 4 x 4 instructions, so every 16-byte operand read from LDS feeds four instructions (twice the reuse
// of the 64 x 128 wavefront blocks).  The 256 int32 accumulators per lane live in the accumulation registers;
// one workgroup per CU.
template <int KS>
__global__ __launch_bounds__(256, 1) void gemm_i8_tile_kernel(GemmI8Args g) {
  constexpr int BM = 256, BN = 256, LD = KS + 16, SEG = KS / 16;
  constexpr int V = BM * KS / 16 / 256;  // 16-byte vectors of A (and of B) per thread per stage
  __shared__ __attribute__((aligned(16))) int8_t As[2][BM * LD];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][BN * LD];

  constexpr int64_t GM = 8;
  const int64_t tiles_n = g.n / BN, tiles_m = g.m / BM, tiles = tiles_m * tiles_n;
  int64_t tile = blockIdx.x;
  if ((tiles & 7) == 0) tile = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int64_t group = tile / (GM * tiles_n);
  const int64_t first_m = group * GM;
  const int64_t gsize = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
  const int64_t within = tile - group * GM * tiles_n;
  const int64_t row0 = (first_m + within % gsize) * BM, col0 = (within / gsize) * BN;

  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int ar = 128 * wr + (lane & 31), bc = 128 * wc + (lane & 31);
  const int kh = 16 * (lane >> 5);
  // this thread's global sources and LDS slots: vector idx = t + 256 it is row idx / SEG, segment idx % SEG
  const int8_t* ga[V];
  const int8_t* gb[V];
  int so[V];
#pragma unroll
  for (int it = 0; it < V; ++it) {
    const int idx = t + 256 * it, r = idx / SEG, sg = idx % SEG;
    ga[it] = g.a + (row0 + r) * g.lda + 16 * sg;
    gb[it] = g.b + (col0 + r) * g.ldb + 16 * sg;
    so[it] = r * LD + 16 * sg;
  }

  i32x16 acc[4][4];
#pragma unroll
  for (int h = 0; h < 4; ++h)
#pragma unroll
    for (int v2 = 0; v2 < 4; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[h][v2][v] = 0;

  const int64_t ns = g.k / KS;
  {
    i32x4 ra[V], rb[V];
#pragma unroll
    for (int it = 0; it < V; ++it) {
      ra[it] = *reinterpret_cast<const i32x4*>(ga[it]);
      rb[it] = *reinterpret_cast<const i32x4*>(gb[it]);
    }
#pragma unroll
    for (int it = 0; it < V; ++it) {
      *reinterpret_cast<i32x4*>(As[0] + so[it]) = ra[it];
      *reinterpret_cast<i32x4*>(Bs[0] + so[it]) = rb[it];
    }
  }
  __syncthreads();
  // stage s's multiply-adds from LDS buffer s & 1
  auto compute = [&](int buf) {
    const int8_t* as = As[buf];
    const int8_t* bs = Bs[buf];
#pragma unroll
    for (int ks = 0; ks < KS / 32; ++ks) {
      const int kk = 32 * ks + kh;
      i32x4 a[4], b[4];
#pragma unroll
      for (int h = 0; h < 4; ++h) a[h] = *reinterpret_cast<const i32x4*>(as + (ar + 32 * h) * LD + kk);
#pragma unroll
      for (int v2 = 0; v2 < 4; ++v2) b[v2] = *reinterpret_cast<const i32x4*>(bs + (bc + 32 * v2) * LD + kk);
#pragma unroll
      for (int h = 0; h < 4; ++h)
#pragma unroll
        for (int v2 = 0; v2 < 4; ++v2)
          acc[h][v2] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[h], b[v2], acc[h][v2], 0, 0, 0);
    }
  };
  for (int64_t s = 0; s + 1 < ns; ++s) {
    const int buf = (int)(s & 1);
    const int64_t off = (s + 1) * KS;
    i32x4 ra[V], rb[V];
#pragma unroll
    for (int it = 0; it < V; ++it) {
      ra[it] = *reinterpret_cast<const i32x4*>(ga[it] + off);
      rb[it] = *reinterpret_cast<const i32x4*>(gb[it] + off);
    }
    __builtin_amdgcn_sched_barrier(0);
    compute(buf);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int it = 0; it < V; ++it) {
      *reinterpret_cast<i32x4*>(As[buf ^ 1] + so[it]) = ra[it];
      *reinterpret_cast<i32x4*>(Bs[buf ^ 1] + so[it]) = rb[it];
    }
    __syncthreads();
  }
  compute((int)((ns - 1) & 1));

  // result layout: register v, lane l -> row (v % 4) + 4 (l / 32) + 8 (v / 4), column l % 32 of the block.
  // The wavefront-uniform part of each address (block, row within the lane group) is kept apart from the
  // lane's offset, so the stores take a scalar base and a 32-bit lane offset.
  const int64_t wrow = row0 + 128 * wr, wcol = col0 + 128 * wc;
  const int lo = 4 * (lane >> 5) * (int)g.ldc + (lane & 31);  // the launcher keeps 260 ldc below 2^31
  if (g.y) {
    const float sa = *g.sa;
#pragma unroll
    for (int v2 = 0; v2 < 4; ++v2) {
      const float sbj = g.sb[g.sb_scalar ? 0 : wcol + 32 * v2 + (lane & 31)];
#pragma unroll
      for (int h = 0; h < 4; ++h)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          float* Yr = g.y + (wrow + 32 * h + (v & 3) + 8 * (v >> 2)) * g.ldc + wcol + 32 * v2;
          const float af = (float)acc[h][v2][v];  // round to nearest even
          const float tq = af * sa;
          Yr[lo] = tq * sbj;
          if ((v & 3) == 3) __builtin_amdgcn_sched_barrier(0);  // a few accumulators at a time
        }
    }
  }
  if (g.acc) {
#pragma unroll
    for (int v2 = 0; v2 < 4; ++v2)
#pragma unroll
      for (int h = 0; h < 4; ++h)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          int32_t* Ar = g.acc + (wrow + 32 * h + (v & 3) + 8 * (v >> 2)) * g.ldc + wcol + 32 * v2;
          Ar[lo] = acc[h][v2][v];
          if ((v & 3) == 3) __builtin_amdgcn_sched_barrier(0);
        }
  }
}

template <int KS>
static hipError_t launch_i8_tile(const GemmI8Args& g, hipStream_t s) {
  const int64_t tiles = (g.m / 256) * (g.n / 256);
  hipLaunchKernelGGL((gemm_i8_tile_kernel<KS>), dim3((unsigned)tiles), dim3(256), 0, s, g);
  return hipGetLastError();
}

template <int HB, int WN, int KS, int NW>
static hipError_t launch_i8(const GemmI8Args& g, hipStream_t s) {
  using Cf = I8Cfg<HB, WN, KS, NW>;
  const int64_t tiles = ((g.m + Cf::BM - 1) / Cf::BM) * ((g.n + Cf::BN - 1) / Cf::BN);
  hipLaunchKernelGGL((gemm_i8_kernel<HB, WN, KS, NW>), dim3((unsigned)tiles), dim3(Cf::NT), 0, s, g);
  return hipGetLastError();
}

hipError_t gemm_i8_launch(const GemmI8Args& gin, hipStream_t s) {
  if (gin.m == 0 || gin.n == 0) return hipSuccess;
  GemmI8Args g = gin;
  g.vec = ((uintptr_t)g.a & 15) == 0 && ((uintptr_t)g.b & 15) == 0 && g.lda % 16 == 0 && g.ldb % 16 == 0;
  // 256 x 256 tiles of 8 wavefronts (one workgroup per CU, 64-byte stages) halve the operand bytes staged per
  // multiply-add and run a tile's work about 1.12x faster than four 128 x 128 tiles of 4 wavefronts (two
  // workgroups per CU); they are taken unless their coarser rounds of workgroups over the CUs cost more
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) !=
                                              hipSuccess || cus <= 0)
    cus = 256;
  const int64_t small_tiles = ((g.m + 127) / 128) * ((g.n + 127) / 128);
  const int64_t big_tiles = ((g.m + 255) / 256) * ((g.n + 255) / 256);
  const double small_time = (double)((small_tiles + 2 * cus - 1) / (2 * cus));        // rounds of one tile time
  const double big_time = (double)((big_tiles + cus - 1) / cus) * (2.0 / 1.12);
  // whole 256 x 256 tiles: the 128 x 128 wavefront blocks (1.06-1.16x the rate of the 64 x 128 blocks at the
  // 1B projection shapes), with 128-byte stages when k allows
  const bool whole = g.vec && g.m % 256 == 0 && g.n % 256 == 0 && g.ldc * 260 < (int64_t(1) << 31);
  if (whole && g.k % 128 == 0) return launch_i8_tile<128>(g, s);
  if (whole && g.k % 64 == 0) return launch_i8_tile<64>(g, s);
  if (big_time < small_time) return launch_i8<2, 4, 64, 8>(g, s);
  return launch_i8<2, 2, 128, 4>(g, s);
}

}  // namespace canon
