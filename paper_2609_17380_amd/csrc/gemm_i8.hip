// gemm_i8.hip - exact int8 GEMM on the int8 matrix cores, with the dequantisation epilogue of the int8
// quantised linear.
//
// acc[i][j] = sum over k of a[i][k] * b[j][k] with int8 operands (a [m][k], b [n][k], both k-contiguous,
// b holding one output column per row as weights [out][in] do).  Integer products and sums are exact, and
// |acc| < 2^31 for k <= 65536, so every summation order gives the same int32: the k loop may be split,
// reordered and spread over matrix instructions freely.  The dequantised output is
// y[i][j] = RN(RN(RN32(acc) * sa) * sb[j]).
//
// Tiling: whole 256 x 256 tiles (m, n multiples of 256, k of 64) run on 4 wavefronts, each a 128 x 128 block of
// 4 x 4 v_mfma_i32_32x32x32_i8 instructions, with direct-to-LDS loads three stages ahead (gemm_i8_tile_kernel).
// Other shapes: a workgroup of NW wavefronts owns a 16 NW HB x 64 WN output tile, each wavefront a 32 HB x 32 WN
// block: 256 x 256 tiles of 8 wavefronts with 64-byte stages for large products, else 128 x 128 tiles of 4
// wavefronts with 128-byte stages; their stages of KS k bytes are staged through registers into LDS (rows
// padded by 16 bytes, which keeps the 16-byte operand reads of 32 consecutive rows free of bank conflicts),
// double buffered.
// Each lane of a 32x32x32 instruction supplies 16 consecutive k bytes of one row of A and of B; the two
// half-wavefronts cover k 0..15 and 16..31 of the instruction's 32.
#include <hip/hip_runtime.h>

#include <type_traits>

#include "canon_internal.h"

namespace canon {

typedef int32_t i32x4 __attribute__((ext_vector_type(4)));
typedef int32_t i32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

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

// 16 bytes per lane from global memory straight into LDS: lane l of the wavefront writes lds_addr + 16 l
// (lds_addr wavefront-uniform, in m0).  Written as assembly so that the compiler does not track these loads:
// it would otherwise wait for all of them before every LDS read, which defeats loading stages ahead; the
// kernel waits for them itself (vm_wait).  The kernel issues no other instruction that uses m0.
#pragma clang diagnostic push
#pragma clang diagnostic ignored "-Winline-asm"
__device__ __forceinline__ void dma16(const int8_t* g, unsigned lds_addr) {
  asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, off" ::"s"(lds_addr), "v"(g)
               : "memory", "m0");
}
#pragma clang diagnostic pop
// wait until at most N vector-memory loads of this wavefront are outstanding (they complete in order)
template <int N>
__device__ __forceinline__ void vm_wait() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);  // expcnt, lgkmcnt left at max
}

// Whole 256 x 256 tiles (m, n multiples of 256, k of 64, 16-byte aligned rows), one workgroup per CU.  NW = 4:
// 4 wavefronts, each a 128 x 128 block of 4 x 4 instructions (256 int32 accumulators per lane), one per SIMD.
// NW = 8 (used): 8 wavefronts, each 128 x 64 as 4 x 2 instructions (128 accumulators), two per SIMD, so one
// wavefront's direct loads, barrier and LDS waits overlap the other's products (15% faster at k = 2048; LDS
// reads, 50% more per product, stay well under the CU's LDS bandwidth).  The pipeline:
//  * stages of 64 k bytes go from global memory straight into LDS (16-byte direct-to-LDS loads, no register
//    staging), NBUF = 4 stages deep: stage s + 3 is requested while stage s is multiplied;
//  * LDS rows are 64 bytes with their four 16-byte segments permuted by the row (segment c of row r at
//    position c ^ sw(r), sw(r) = ((r >> 2) ^ (r & 2)) & 3), so the operand reads of 8 (or 16) consecutive
//    rows at one k offset cover distinct banks; each direct load of a wavefront fills 16 rows, lane l the
//    position l of that kilobyte, fetching the global segment that belongs there;
//  * operand fragments run one k step ahead (two sets), and the stage's barrier sits before the last k
//    step's instructions, whose fragments are already in registers.
// Buffer safety: buffer (s + 3) % NBUF = (s - 1) % NBUF is refilled during stage s, after the barrier inside
// stage s - 1, which every wavefront passes only once its reads of stage s - 1 have completed; stage s + 1 is
// read after the barrier inside stage s, which every wavefront passes only once its own loads of stage s + 1
// have landed.
// NW = 8: eight wavefronts (two per SIMD), each a 128 x 64 block of 4 x 2 instructions (128 accumulators), four
// direct loads per wavefront and stage.
template <int NBUF, int NW>
__global__ __launch_bounds__(64 * NW, 1) void gemm_i8_tile_kernel(GemmI8Args g) {
  constexpr int BM = 256, BN = 256, KS = 64, ROWB = 64;
  constexpr int STAGE = (BM + BN) * KS;  // bytes per stage: A rows, then B rows
  static_assert(NBUF == 4, "three stages ahead: the waits below count three");
  static_assert(NW == 4 || NW == 8, "four or eight wavefronts");
  constexpr int WC = NW / 2, WCOLS = BN / WC, V2N = WCOLS / 32;  // wavefront columns, its width, its 32-col blocks
  constexpr int RB = 16 / NW;   // 16-row blocks of A (and of B) each wavefront loads per stage
  constexpr int LPW = 2 * RB;   // direct loads per wavefront and stage
  __shared__ __attribute__((aligned(1024))) int8_t lds[NBUF * STAGE];

  constexpr int64_t GM = 8;
  const int64_t tiles_n = g.n / BN, tiles_m = g.m / BM, tiles = tiles_m * tiles_n;
  int64_t tile = blockIdx.x;
  if ((tiles & 7) == 0) tile = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int64_t group = tile / (GM * tiles_n);
  const int64_t first_m = group * GM;
  const int64_t gsize = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
  const int64_t within = tile - group * GM * tiles_n;
  const int64_t row0 = (first_m + within % gsize) * BM, col0 = (within / gsize) * BN;

  const int t = threadIdx.x, lane = t & 63;
  const int w = __builtin_amdgcn_readfirstlane(t >> 6);
  const int wr = w / WC, wc = w % WC;
  // fragment reads: lane (rl, hi) reads row rl of a 32-row block at k segment 2 ks + hi
  const int rl = lane & 31, hi = lane >> 5;
  const int cs = hi ^ (((rl >> 2) ^ (rl & 2)) & 3);
  const int seg0 = 16 * cs, seg1 = 16 * (cs ^ 2);  // positions of segments hi and 2 + hi
  const int a_off = (128 * wr + rl) * ROWB, b_off = BM * KS + (WCOLS * wc + rl) * ROWB;
  // direct loads: wavefront w fills row blocks RB w .. RB w + RB - 1 (16 rows each) of A and of B; lane l writes
  // position l of a block: row l / 4, segment position l % 4, holding global segment (l % 4) ^ sw(row)
  const int dr = lane >> 2;
  const int dseg = (lane & 3) ^ (((dr >> 2) ^ (dr & 2)) & 3);
  const int8_t* ga = g.a + (row0 + 16 * RB * w + dr) * g.lda + 16 * dseg;
  const int8_t* gb = g.b + (col0 + 16 * RB * w + dr) * g.ldb + 16 * dseg;
  const int64_t sta = 16 * g.lda, stb = 16 * g.ldb;

  i32x16 acc[4][V2N];
#pragma unroll
  for (int h = 0; h < 4; ++h)
#pragma unroll
    for (int v2 = 0; v2 < V2N; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[h][v2][v] = 0;

  const int64_t ns = g.k / KS;
  i32x4 fa[2][4], fb[2][V2N];  // two fragment sets
  // wavefront-uniform LDS byte address of this wavefront's first row block in stage buffer 0
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) int8_t*)lds + 16 * RB * w * ROWB;
  auto issue = [&](int64_t st) {
    const unsigned base = lds0 + (unsigned)(st & (NBUF - 1)) * STAGE;
    const int64_t k0 = st * KS;
#pragma unroll
    for (int i = 0; i < RB; ++i) {
      dma16(ga + i * sta + k0, base + 16 * i * ROWB);
      dma16(gb + i * stb + k0, base + BM * KS + 16 * i * ROWB);
    }
  };
  auto frags = [&](int f, int64_t st, int ks) {
    const int8_t* base = lds + (int)(st & (NBUF - 1)) * STAGE;
    const int so = ks ? seg1 : seg0;
#pragma unroll
    for (int h = 0; h < 4; ++h) fa[f][h] = *reinterpret_cast<const i32x4*>(base + a_off + 32 * h * ROWB + so);
#pragma unroll
    for (int v2 = 0; v2 < V2N; ++v2) fb[f][v2] = *reinterpret_cast<const i32x4*>(base + b_off + 32 * v2 * ROWB + so);
  };
  auto mma = [&](int f) {
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int v2 = 0; v2 < V2N; ++v2)
        acc[h][v2] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[f][h], fb[f][v2], acc[h][v2], 0, 0, 0);
  };

  issue(0);
  if (ns > 1) issue(1);
  if (ns > 2) issue(2);
  // stage 0 landed (this wavefront's loads of stages 1 and 2 may still be in flight), then everyone's
  if (ns > 2) vm_wait<2 * LPW>();
  else if (ns > 1) vm_wait<LPW>();
  else vm_wait<0>();
  __syncthreads();
  frags(0, 0, 0);
  // Every stage but the last: no branch around LDS operations inside the loop, so the compiler's wait counts
  // stay exact (the last k step's instructions wait only for their own fragments, not for the next stage's
  // reads issued after the barrier).
  // k step 0 of a stage with the LPW loads of stage st + 3 spread over its 4 V2N instructions (one load after
  // every two): issued in one burst they stall the wavefront while the matrix core idles
  auto mma0_loads = [&](int64_t st3, bool more) {  // more: stage st3 exists (wavefront-uniform)
    const unsigned base = lds0 + (unsigned)(st3 & (NBUF - 1)) * STAGE;
    const int64_t k0 = st3 * KS;
#pragma unroll
    for (int h = 0; h < 4; ++h)
#pragma unroll
      for (int v2 = 0; v2 < V2N; ++v2) {
        acc[h][v2] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[0][h], fb[0][v2], acc[h][v2], 0, 0, 0);
        if (v2 & 1) {
          const int j = (h * V2N + v2) >> 1, i = j >> 1, ab = j & 1;  // pieces in order A0, B0, A1, B1, ...
          if (more) {
            if (ab == 0) dma16(ga + i * sta + k0, base + 16 * i * ROWB);
            else dma16(gb + i * stb + k0, base + BM * KS + 16 * i * ROWB);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
  };
  for (int64_t st = 0; st + 1 < ns; ++st) {
    frags(1, st, 1);
    mma0_loads(st + 3, st + 3 < ns);
    __builtin_amdgcn_sched_barrier(0);
    // this wavefront's loads of stage st + 1 landed (those of later stages may stay in flight), then everyone's
    if (st + 3 < ns) vm_wait<2 * LPW>();
    else if (st + 2 < ns) vm_wait<LPW>();
    else vm_wait<0>();
    __syncthreads();
    frags(0, st + 1, 0);
    mma(1);
    // the next stage's reads first, under this step's 16 instructions
    __builtin_amdgcn_sched_group_barrier(0x100, 4 + V2N, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 4 * V2N, 0);
    __builtin_amdgcn_sched_barrier(0);
  }
  frags(1, ns - 1, 1);
  mma(0);
  mma(1);

  // Epilogue through LDS, 32 rows of the wavefront's 128 x WCOLS block at a time, so that every lane stores 16
  // contiguous bytes (4 columns) and a store instruction covers 64 / (WCOLS / 4) row segments of 4 WCOLS bytes.  Result layout of
  // the instruction: register v, lane (rl, hi) -> row (v % 4) + 4 hi + 8 (v / 4), column rl of the 32 x 32
  // block.  Each wavefront writes and reads back only its own LDS region (LDS operations of a wavefront complete
  // in order); the barrier first lets every wavefront finish reading the last stage.
  constexpr int ELD = WCOLS + 8;  // padded row (ints): the two half-wavefronts' rows 4 apart fall on other banks
  constexpr int LPR = WCOLS / 4, RPI = 64 / LPR;  // read-back lanes per row, rows per instruction
  static_assert(NW * 32 * ELD * 4 <= NBUF * STAGE, "epilogue rows fit in the stage buffers");
  __syncthreads();
  int32_t* eb = reinterpret_cast<int32_t*>(lds) + w * (32 * ELD);
  const int64_t wrow = row0 + 128 * wr, wcol = col0 + WCOLS * wc;
  const int c4 = 4 * (lane % LPR), rq = lane / LPR;  // this lane's 4 columns and row offset in the read-back
  float sa = 0.0f, sb4[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  if (g.y) {
    sa = *g.sa;
#pragma unroll
    for (int e = 0; e < 4; ++e) sb4[e] = g.sb[g.sb_scalar ? 0 : wcol + c4 + e];
  }
#pragma unroll
  for (int h = 0; h < 4; ++h) {
#pragma unroll
    for (int v2 = 0; v2 < V2N; ++v2)
#pragma unroll
      for (int v = 0; v < 16; ++v) eb[((v & 3) + 4 * hi + 8 * (v >> 2)) * ELD + 32 * v2 + rl] = acc[h][v2][v];
#pragma unroll
    for (int q = 0; q < 32 / RPI; ++q) {
      const int r = RPI * q + rq;
      const i32x4 x = *reinterpret_cast<const i32x4*>(eb + r * ELD + c4);
      const int64_t o = (wrow + 32 * h + r) * g.ldc + wcol + c4;
      if (g.y) {  // streamed out: nontemporal
        f32x4 y;
        y[0] = ((float)x[0] * sa) * sb4[0];  // RN(RN(RN32(acc) sa) sb), one rounding per operation
        y[1] = ((float)x[1] * sa) * sb4[1];
        y[2] = ((float)x[2] * sa) * sb4[2];
        y[3] = ((float)x[3] * sa) * sb4[3];
        __builtin_nontemporal_store(y, reinterpret_cast<f32x4*>(g.y + o));
      }
      if (g.acc) __builtin_nontemporal_store(x, reinterpret_cast<i32x4*>(g.acc + o));
    }
  }
}

constexpr int kI8TileWaves = 8;

static hipError_t launch_i8_tile(const GemmI8Args& g, hipStream_t s) {
  const int64_t tiles = (g.m / 256) * (g.n / 256);
  hipLaunchKernelGGL((gemm_i8_tile_kernel<4, kI8TileWaves>), dim3((unsigned)tiles), dim3(64 * kI8TileWaves), 0, s, g);
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
  // whole 256 x 256 tiles (and 16-byte output stores: y, acc and ldc aligned to 4 elements): the pipelined
  // kernel with 128 x 128 wavefront blocks
  const bool whole = g.vec && g.m % 256 == 0 && g.n % 256 == 0 && g.ldc % 4 == 0 && ((uintptr_t)g.y & 15) == 0 &&
                     ((uintptr_t)g.acc & 15) == 0;
  if (whole && g.k % 64 == 0 && g.k > 0) return launch_i8_tile(g, s);
  if (big_time < small_time) return launch_i8<2, 4, 64, 8>(g, s);
  return launch_i8<2, 2, 128, 4>(g, s);
}

}  // namespace canon
