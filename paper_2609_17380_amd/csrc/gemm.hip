// gemm.hip - canonical-order GEMM (R1, R2) on gfx950 matrix cores.
//
// C[i,j] = sum_k A(i,k) B(k,j): the k terms form chunks of 32; each chunk is a left-to-right chain of
// fused multiply-adds from +0 in ascending k; the chunk partials are combined by the binary-carry fold of
// Algorithm 2 (pushed in ascending chunk order, leftover blocks combined smallest first).
//
// Matrix-core mapping.  v_mfma_f32_32x32x1_2b_f32 (two independent 32x32 blocks) and
// v_mfma_f32_16x16x1_4b_f32 (four 16x16 blocks) perform the rank-1 update D = C + a*b with ONE product per
// output element.  On gfx950 they return RN(c + a*b) with the flush rule of R0, bit for bit (checked against
// a sequential fma chain, including ties, signed zeros and 32-step dependent chains).  A bf16 x bf16 product
// is exact in fp32, so a chain of these updates, one per k, is exactly the canonical fma chain.  The bf16
// MFMA shapes that sum several products inside one instruction do not give the chain's roundings and are
// not used.
//
// Tiling (GemmCfg): a workgroup computes a 64-row tile of C, 128 columns with four wavefronts of the 32x32
// instruction (wave (wr, wc) owns rows 32*wr..+32 and columns 64*wc..+64 as two 32x32 blocks), or 64 columns
// with four wavefronts of the 16x16 instruction (wave w owns rows 16*w..+16 as four 16x16 blocks).  Two or
// three workgroups share a CU so one hides the others' LDS and barrier waits.  Per chunk the 64x32 A tile and
// the 32-deep B tile are staged through LDS as fp32, widened once and double buffered, with the next chunk's
// 16-byte global loads in flight during the current chunk's MFMA chain.  An operand whose source is
// k-contiguous is stored as rows [row][k] (one 16-byte LDS read gives a lane four k values); one whose source
// is row-contiguous is either stored k-major [k][row] (one 4-byte read per k, no transposing scatter) or, in
// the shapes that read twice as often, scattered into rows with a bank-spreading permutation (LROWX).
// Fold: inside an aligned group of four chunks the two lowest levels of Algorithm 2 are fixed and merged
// in place; the group partial is pushed at level 2.  The next levels (2 to 4 of them, by shape) stay in
// registers; the levels above, touched once per 16 chunks or less often, live in per-lane private memory.
//
// Causal modes (attention): KMODE_TRAIL skips key chunks that are masked for every row of the tile and
// KMODE_LEAD skips query chunks below the tile; the skipped chunks' partials are exactly +0 in the
// canonical chain and are still folded (pushed as +0), so the result equals the full-range chain.  With a
// sliding window kwin, TRAIL also skips the key chunks before the window of the tile's first query and
// LEAD the query chunks after the window of the tile's last key.  Output tiles with no visible entry
// (tri_lower: above the diagonal, or left of the window band) are not computed: the dS epilogue writes
// their +0 (every such tile when zero_dead, else the band tiles within the readers' reach, kAttnLead),
// other outputs leave them unwritten.
#include <hip/hip_runtime.h>

#include "canon_dev.h"
#include "canon_internal.h"

namespace canon {

typedef float v32f __attribute__((ext_vector_type(32)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v16f __attribute__((ext_vector_type(16)));

// The rank-1 matrix instructions; both add exactly one product into every output.  V = 32:
// v_mfma_f32_32x32x1_2b_f32, a wavefront owns 32 x 64 outputs (two 32x32 blocks sharing the A column), 32
// accumulators per lane.  V = 16: v_mfma_f32_16x16x1_4b_f32, a wavefront owns 16 x 64 (four 16x16 blocks sharing
// the A column), 16 accumulators per lane: half the registers per chain and per fold level.
template <int V>
struct Mfma;
template <>
struct Mfma<32> {
  typedef v32f T;
  static constexpr int WR = 32;  // rows per wavefront
  static __device__ __forceinline__ T step(float a, float b, const T& c) {
    return __builtin_amdgcn_mfma_f32_32x32x1f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ int arow(int lane) { return lane & 31; }  // A row of this lane
  // output register v of a lane -> row and column inside the wavefront's block
  static __device__ __forceinline__ int orow(int v, int lane) {
    return (v & 3) + 4 * (lane >> 5) + 8 * ((v & 15) >> 2);
  }
  static __device__ __forceinline__ int ocol(int v, int lane) { return (v >> 4) * 32 + (lane & 31); }
};
template <>
struct Mfma<16> {
  typedef v16f T;
  static constexpr int WR = 16;
  static __device__ __forceinline__ T step(float a, float b, const T& c) {
    return __builtin_amdgcn_mfma_f32_16x16x1f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ int arow(int lane) { return lane & 15; }
  static __device__ __forceinline__ int orow(int v, int lane) { return (v & 3) + 4 * (lane >> 4); }
  static __device__ __forceinline__ int ocol(int v, int lane) { return (v >> 2) * 16 + (lane & 15); }
};

constexpr int BM = 64, BN = 128, KC = 32;
static_assert(BM <= 128 && 128 % BM == 0 && KC == 32, "the attention read reach (kAttnLead) assumes these tiles");
constexpr int LDK = KC + 4;               // row-layout stride (floats): [row][k]
constexpr int LDMA = BM + 4, LDMB = BN + 4;  // k-major stride (floats): [k][row]
constexpr int A_FLOATS = (BM * LDK > KC * LDMA) ? BM * LDK : KC * LDMA;
constexpr int B_FLOATS = (BN * LDK > KC * LDMB) ? BN * LDK : KC * LDMB;

// Workgroup shape of the general kernel: instruction V, WC wavefront columns of 64 (the tile is 64 x 64*WC, the
// wavefronts (64 / WR) x WC), OCC workgroups per CU, the number of fold levels kept in registers for the
// row/row layout (RLR) and the layouts with a k-major operand (RLK), and TR: a k-major operand is transposed
// while it is staged, so that every chain read is a 16-byte row read.
template <int V_, int WC_, int OCC_, int RLR_, int RLK_, bool TR_ = false>
struct GemmCfg {
  static constexpr int V = V_, WC = WC_, OCC = OCC_, RLR = RLR_, RLK = RLK_;
  static constexpr bool TR = TR_;
  static constexpr int NW = (BM / Mfma<V>::WR) * WC, NT = 64 * NW, TBN = 64 * WC, LDMB = TBN + 4;
  static constexpr int BFL = (TBN * LDK > KC * LDMB) ? TBN * LDK : KC * LDMB;
};

// Layout of an operand tile in LDS: LROW [row][k] (stride LDK); LKM k-major [k][row] (stride LDM); LROWX
// [row][k] with the 16-byte k segments of row r permuted by r: element (r, k) at r * LDK + (k ^ swz(r)).  LROWX
// holds transposed k-major sources: the staging thread writes one k of eight consecutive rows, and the permutation
// (constant over those rows) spreads the eight rows of a wavefront's writes over distinct banks.
enum { LROW = 0, LKM = 1, LROWX = 2 };
__device__ __forceinline__ int swz(int r) { return 4 * ((r >> 4) & 7); }

// Raw bf16 data of one chunk for one thread: 8 A elements and 16 B elements, as 16-byte vectors.
struct Raw {
  uint4 a, b0, b1;
};

// bf16 pair packed in a 32-bit word -> two floats.  No explicit input flush: in flush mode the matrix
// core reads a subnormal operand as zero of its sign (measured on gfx950), which is the R0 input rule.
__device__ __forceinline__ void widen8(const uint4& u, float (&f)[8]) {
  f[0] = __uint_as_float(u.x << 16); f[1] = __uint_as_float(u.x & 0xFFFF0000u);
  f[2] = __uint_as_float(u.y << 16); f[3] = __uint_as_float(u.y & 0xFFFF0000u);
  f[4] = __uint_as_float(u.z << 16); f[5] = __uint_as_float(u.z & 0xFFFF0000u);
  f[6] = __uint_as_float(u.w << 16); f[7] = __uint_as_float(u.w & 0xFFFF0000u);
}

__device__ __forceinline__ uint4 pack8(const uint16_t (&h)[8]) {
  uint4 u;
  u.x = (uint32_t)h[0] | ((uint32_t)h[1] << 16);
  u.y = (uint32_t)h[2] | ((uint32_t)h[3] << 16);
  u.z = (uint32_t)h[4] | ((uint32_t)h[5] << 16);
  u.w = (uint32_t)h[6] | ((uint32_t)h[7] << 16);
  return u;
}

// 8 consecutive elements of which only the first `valid` exist: zero fill beyond.
template <bool FAST>
__device__ __forceinline__ uint4 load8(const uint16_t* p, int64_t valid, bool vec) {
  if (FAST) return *reinterpret_cast<const uint4*>(p);
  if (vec && valid >= 8) return *reinterpret_cast<const uint4*>(p);
  uint16_t h[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) h[e] = (e < valid) ? p[e] : (uint16_t)0;
  return pack8(h);
}

// Global -> registers for the chunk starting at k0.  Per operand, a thread takes 8 consecutive elements
// along the source's contiguous dimension: (row, 8 k) for a k-contiguous source, (k, 8 rows) otherwise.
// FAST: the whole chunk is in range and 16-byte aligned (no checks).
template <bool TA, bool TB, bool FAST, int NT, int TBN>
__device__ __forceinline__ Raw load_chunk(const GemmArgs& g, const uint16_t* A, const uint16_t* B, int64_t row0,
                                          int64_t col0, int64_t k0, bool vec) {
  const int t = threadIdx.x;
  Raw r;
  if (NT == 256 || t < 256) {  // 256 A pieces
    if (!TA) {
      const int64_t row = row0 + (t >> 2), k = k0 + (t & 3) * 8;
      r.a = load8<FAST>(A + row * g.lda + k, (row < g.m) ? (g.k - k) : 0, vec);
    } else {
      const int64_t k = k0 + (t >> 3), row = row0 + (t & 7) * 8;
      r.a = load8<FAST>(A + k * g.lda + row, (k < g.k) ? (g.m - row) : 0, vec);
    }
  }
#pragma unroll
  for (int it = 0; it < 4 * TBN / NT; ++it) {  // 4 * TBN B pieces
    const int idx = t + NT * it;
    uint4 v;
    if (TB) {
      const int64_t col = col0 + (idx >> 2), k = k0 + (idx & 3) * 8;
      v = load8<FAST>(B + col * g.ldb + k, (col < g.n) ? (g.k - k) : 0, vec);
    } else {
      const int64_t k = k0 + idx / (TBN / 8), col = col0 + (idx % (TBN / 8)) * 8;
      v = load8<FAST>(B + k * g.ldb + col, (k < g.k) ? (g.n - col) : 0, vec);
    }
    if (it == 0) r.b0 = v; else r.b1 = v;
  }
  return r;
}

__device__ __forceinline__ void st8(float* d, const float (&f)[8]) {
  *reinterpret_cast<v4f*>(d) = v4f{f[0], f[1], f[2], f[3]};
  *reinterpret_cast<v4f*>(d + 4) = v4f{f[4], f[5], f[6], f[7]};
}

// Registers -> LDS: rows [row][k] for k-contiguous sources, k-major [k][row] otherwise; both are
// 8 contiguous floats per thread.
// one k of eight consecutive rows r0.. into an LROWX tile
__device__ __forceinline__ void st8x(float* d, int r0, int k, const float (&f)[8]) {
  const int kx = k ^ swz(r0);  // r0 is a multiple of 8: the eight rows share swz
#pragma unroll
  for (int e = 0; e < 8; ++e) d[(r0 + e) * LDK + kx] = f[e];
}

template <bool TA, bool TB, int NT, int TBN, bool TR = false>
__device__ __forceinline__ void store_chunk(float* As, float* Bs, const Raw& r) {
  const int t = threadIdx.x;
  float f[8];
  if (NT == 256 || t < 256) {
    widen8(r.a, f);
    if (!TA) st8(As + (t >> 2) * LDK + (t & 3) * 8, f);
    else if (TR) st8x(As, (t & 7) * 8, t >> 3, f);
    else st8(As + (t >> 3) * LDMA + (t & 7) * 8, f);
  }
#pragma unroll
  for (int it = 0; it < 4 * TBN / NT; ++it) {
    const int idx = t + NT * it;
    widen8(it == 0 ? r.b0 : r.b1, f);
    if (TB) st8(Bs + (idx >> 2) * LDK + (idx & 3) * 8, f);
    else if (TR) st8x(Bs, (idx % (TBN / 8)) * 8, idx / (TBN / 8), f);
    else st8(Bs + (idx / (TBN / 8)) * (TBN + 4) + (idx % (TBN / 8)) * 8, f);
  }
}

// four consecutive k values (4*g4 .. 4*g4+3) of this lane's row / column
template <int L, int LDM>
__device__ __forceinline__ v4f fetch4(const float* base, int idx, int g4) {
  if (L == LROW) return *reinterpret_cast<const v4f*>(base + idx * LDK + 4 * g4);
  if (L == LROWX) return *reinterpret_cast<const v4f*>(base + idx * LDK + ((4 * g4) ^ swz(idx)));
  const float* p = base + (4 * g4) * LDM + idx;
  return v4f{p[0], p[LDM], p[2 * LDM], p[3 * LDM]};
}
// the single value (idx, kk)
template <int L, int LDM>
__device__ __forceinline__ float elem(const float* base, int idx, int kk) {
  if (L == LROW) return base[idx * LDK + kk];
  if (L == LROWX) return base[idx * LDK + (kk ^ swz(idx))];
  return base[kk * LDM + idx];
}
// the LDS layout of an operand: transposed (TA for A, !TB for B) sources are k-major unless TR
template <bool TRANSPOSED, bool TR>
struct Lay {
  static constexpr int L = !TRANSPOSED ? LROW : (TR ? LROWX : LKM);
};

// One full chunk's chain: 32 dependent rank-1 updates from +0, operand reads one group ahead.
template <bool TA, bool TB, int V, int LDB, bool TR = false>
__device__ __forceinline__ typename Mfma<V>::T chain_full(const float* As, const float* Bs, int ai, int bi) {
  constexpr int LA = Lay<TA, TR>::L, LB = Lay<!TB, TR>::L;
  typename Mfma<V>::T acc;
#pragma unroll
  for (int v = 0; v < V; ++v) acc[v] = 0.0f;
  v4f a4 = fetch4<LA, LDMA>(As, ai, 0), b4 = fetch4<LB, LDB>(Bs, bi, 0);
#pragma unroll
  for (int g4 = 0; g4 < KC / 4; ++g4) {
    v4f an = a4, bn = b4;
    if (g4 + 1 < KC / 4) {
      an = fetch4<LA, LDMA>(As, ai, g4 + 1);
      bn = fetch4<LB, LDB>(Bs, bi, g4 + 1);
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) acc = Mfma<V>::step(a4[j], b4[j], acc);
    a4 = an;
    b4 = bn;
  }
  return acc;
}

// A ragged last chunk: only its kleft < 32 real terms enter the chain.
template <bool TA, bool TB, int V, int LDB, bool TR = false>
__device__ __forceinline__ typename Mfma<V>::T chain_part(const float* As, const float* Bs, int ai, int bi,
                                                          int kleft) {
  constexpr int LA = Lay<TA, TR>::L, LB = Lay<!TB, TR>::L;
  typename Mfma<V>::T acc;
#pragma unroll
  for (int v = 0; v < V; ++v) acc[v] = 0.0f;
  for (int kk = 0; kk < kleft; ++kk) {
    const float av = elem<LA, LDMA>(As, ai, kk);
    const float bv = elem<LB, LDB>(Bs, bi, kk);
    acc = Mfma<V>::step(av, bv, acc);
  }
  return acc;
}

// Fold levels kept in private memory (levels >= the register levels); rarely touched.
template <int N, class T>
struct FoldMem {
  static constexpr int V = sizeof(T) / sizeof(float);
  float s[N > 0 ? N : 1][V];
  // levels whose bit is set in c0 hold +0 (skipped leading blocks); the others are written before read
  __device__ __forceinline__ void clear(int64_t c0) {
    for (int L = 0; L < N; ++L, c0 >>= 1)
      if (c0 & 1)
        for (int v = 0; v < V; ++v) s[L][v] = 0.0f;
  }
  __device__ __forceinline__ void push(T p, int64_t c) {
    int L = 0;
    while (c & 1) {
      T lower;
#pragma unroll
      for (int v = 0; v < V; ++v) lower[v] = s[L][v];
      p = lower + p;
      c >>= 1;
      ++L;
    }
#pragma unroll
    for (int v = 0; v < V; ++v) s[L][v] = p[v];
  }
  __device__ __forceinline__ void result(T& r, bool& have, int64_t n) const {
    for (int L = 0; L < N; ++L, n >>= 1) {
      if (n & 1) {
        T x;
#pragma unroll
        for (int v = 0; v < V; ++v) x[v] = s[L][v];
        if (!have) { r = x; have = true; }
        else r = x + r;
      }
    }
  }
};

// Binary-carry stack of Algorithm 2: R register levels, then the private-memory levels (a separate object,
// so that the dynamically indexed memory levels never force the register levels out of registers).
// push(p, c, mem) pushes the partial with index c at this level: at each level whose bit of c is set the
// stored block is merged (earlier block on the left) and the carry moves up.  The caller keeps the chunk
// count below 2^MAXL.
template <int R, class T>
struct FoldRegs {
  T s;
  FoldRegs<R - 1, T> up;
  // the stack after c0 pushes of +0: +0 at the set bits of c0
  template <class M>
  __device__ __forceinline__ void clear(const T& z, int64_t c0, M& mem) {
    s = z;
    up.clear(z, c0 >> 1, mem);
  }
  template <class M>
  __device__ __forceinline__ void push(T p, int64_t c, M& mem) {
    if (c & 1) up.push(s + p, c >> 1, mem);
    else s = p;
  }
  // push(a + b, c), with the sum formed at the level where the carry stops, so that it is computed straight
  // into that level's registers (no copy)
  template <class M>
  __device__ __forceinline__ void push_sum(const T& a, const T& b, int64_t c, M& mem) {
    if (c & 1) up.push_sum(s, a + b, c >> 1, mem);
    else s = a + b;
  }
  // Result: lowest occupied level first, then the others in ascending level order
  template <class M>
  __device__ __forceinline__ void result(T& r, bool& have, int64_t n, const M& mem) const {
    if (n & 1) {
      if (!have) { r = s; have = true; }
      else r = s + r;
    }
    up.result(r, have, n >> 1, mem);
  }
};
template <class T>
struct FoldRegs<0, T> {
  template <class M>
  __device__ __forceinline__ void clear(const T&, int64_t c0, M& mem) { mem.clear(c0); }
  template <class M>
  __device__ __forceinline__ void push(T p, int64_t c, M& mem) { mem.push(p, c); }
  template <class M>
  __device__ __forceinline__ void push_sum(const T& a, const T& b, int64_t c, M& mem) { mem.push(a + b, c); }
  template <class M>
  __device__ __forceinline__ void result(T& r, bool& have, int64_t n, const M& mem) const {
    mem.result(r, have, n);
  }
};

// CZ: the causal modes, K segments and the triangular output (tri_lower) are compiled in.  Launches with none
// of them (every projection and gradient GEMM) take the CZ = false instantiation, whose chunk loop has no
// skip tests: the same chains and fold, 2.5-5% faster.
template <int MAXL, bool TA, bool TB, class CF, bool CZ>
__global__ __launch_bounds__(CF::NT, CF::OCC * CF::NW / 4) void gemm_mfma_kernel(GemmArgs g) {
  typedef typename Mfma<CF::V>::T vec;
  constexpr int NT = CF::NT, TBN = CF::TBN, V = CF::V, WR = Mfma<V>::WR;
  __shared__ __attribute__((aligned(16))) float As[2][A_FLOATS];
  __shared__ __attribute__((aligned(16))) float Bs[2][CF::BFL];
  // the stack holds levels >= 2 (levels 0 and 1 live inside the group code): register levels (three for
  // the row/row layout, two for layouts with k-major staging, which need more address registers), the
  // rest in private memory
  constexpr int RLMAX = (!TA && TB) ? CF::RLR : CF::RLK;
  constexpr int RL = (MAXL - 2) < RLMAX ? (MAXL - 2) : RLMAX;
  constexpr int NMEM = MAXL - 2 - RL;

  // tile order: consecutive workgroups go to different XCDs, so first give each XCD a contiguous run of
  // tiles; then walk that run in groups of GM tile rows (column of GM tiles, then the next column), so the
  // workgroups resident on one XCD share a few A and B tiles in its L2
  constexpr int64_t GM = 8;
  const int64_t tiles_n = (g.n + TBN - 1) / TBN;
  const int64_t tiles_m = (g.m + BM - 1) / BM;
  const int64_t tiles = tiles_m * tiles_n;
  int64_t tile = blockIdx.x;
  if ((tiles & 7) == 0) tile = (blockIdx.x & 7) * (tiles >> 3) + (blockIdx.x >> 3);
  const int64_t group = tile / (GM * tiles_n);
  const int64_t first_m = group * GM;
  const int64_t gsize = (tiles_m - first_m) < GM ? (tiles_m - first_m) : GM;
  const int64_t within = tile - group * GM * tiles_n;
  int64_t tm = first_m + within % gsize, tn = within / gsize;
  int64_t z = blockIdx.z;
  if (CZ && g.kmode != KMODE_FULL) {
    // causally skipping GEMMs: tile cost grows with the row tile (TRAIL) or shrinks with it (LEAD).  Over the
    // whole launch (in dispatch order, blockIdx.x fastest), the longest tiles of every batch matrix go first
    // so the short ones fill the tail; the batch index runs fastest, so the workgroups on one XCD (every 8th)
    // share its matrices.
    const int64_t l = blockIdx.x + (int64_t)gridDim.x * blockIdx.z;
    const int64_t rank = l / g.batch;
    z = l - rank * g.batch;
    tm = rank / tiles_n;
    tn = rank % tiles_n;
    if (g.kmode == KMODE_TRAIL) tm = tiles_m - 1 - tm;
  }
  const int64_t row0 = tm * BM, col0 = tn * TBN;
  const bool upper_dead = CZ && g.tri_lower && col0 > row0 + BM - 1;                           // above the diagonal
  const bool band_dead = CZ && g.tri_lower && g.kwin > 0 && col0 + TBN - 1 <= row0 - g.kwin;   // left of the window
  // out of every reader's reach (the dS epilogue writes the +0 of the dead tiles the readers reach)
  const bool band_far = band_dead && !g.zero_dead && col0 + TBN - 1 < row0 - g.kwin - kAttnLead;
  if ((upper_dead && !(g.zero_dead && g.epi == EPI_DS)) || (band_dead && (g.epi != EPI_DS || band_far))) return;
  const bool dead = upper_dead || band_dead;  // the epilogue writes this tile's +0

  const int64_t z1 = z / g.nb2, z2 = z % g.nb2;
  const uint16_t* A = g.a + z1 * g.sa1 + z2 * g.sa2;
  const uint16_t* B = g.b + z1 * g.sb1 + (g.b_group > 1 ? z2 / g.b_group : z2) * g.sb2;
  const bool vload = g.vec != 0;
  const bool tile_in = vload && row0 + BM <= g.m && col0 + TBN <= g.n;

  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wr = w / CF::WC, wc = w % CF::WC;
  const int ai = wr * WR + Mfma<V>::arow(lane);  // this lane's A row within the tile
  const int bi = wc * 64 + lane;         // this lane's B column within the tile

  const int64_t nc = (g.k + KC - 1) / KC;
  const int64_t kfull = g.k / KC;  // chunks with all 32 terms
  // The real chunks: in each K segment of spc chunks (one segment unless kseg is set), the local chunks
  // [lb, le); every other chunk is a +0 partial.
  const int64_t spc = (CZ && g.kseg > 0) ? g.kseg / KC : nc;
  const int64_t nseg = (CZ && g.kseg > 0) ? nc / spc : 1;
  const int64_t ncs = (CZ && g.kseg > 0) ? spc : nc;
  int64_t lb = 0, le = ncs;
  const int64_t last_row = row0 + BM < g.m ? row0 + BM : g.m;  // rows of this tile are < last_row
  if (CZ && g.kmode == KMODE_TRAIL) {
    int64_t ce = (last_row + KC - 1) / KC;
    le = ce < ncs ? ce : ncs;
    if (g.kwin > 0 && row0 - g.kwin + 1 > 0) {  // keys before the first query's window
      const int64_t cb = (row0 - g.kwin + 1) / KC;
      lb = cb < le ? cb : le;
    }
  } else if (CZ && g.kmode == KMODE_LEAD) {
    int64_t cb = row0 / KC;
    lb = cb < ncs ? cb : ncs;
    if (g.kwin > 0) {  // queries after the last key's window: the last visible query is last_row - 2 + kwin
      const int64_t ce = (last_row - 2 + g.kwin) / KC + 1;
      le = ce < ncs ? ce : ncs;
      if (le < lb) le = lb;
    }
  }
  if (dead) lb = le = 0;

  vec zero;
#pragma unroll
  for (int v = 0; v < V; ++v) zero[v] = 0.0f;
  // Level-2 stack (one entry per aligned group of four chunks).  Groups entirely before lb (in the first
  // segment) are skipped chunks: pushing them as +0 partials leaves +0 at the set bits of their count,
  // i.e. clear().
  FoldRegs<RL, vec> S;
  FoldMem<NMEM, vec> Smem;
  S.clear(zero, lb >> 2, Smem);

  int buf = 0;
  if (lb < le)
    store_chunk<TA, TB, NT, TBN, CF::TR>(As[0], Bs[0], load_chunk<TA, TB, false, NT, TBN>(g, A, B, row0, col0, lb * KC, vload));
  __syncthreads();

  // generic pipelined chunk (checked loads, ragged chunk allowed): real chunks run in ascending order;
  // nextc is the next real chunk (its loads go ahead of this chunk's chain), or -1
  auto run_chunk = [&](int64_t c, int64_t nextc) -> vec {
    const bool more = nextc >= 0;
    Raw nxt;
    if (more) nxt = load_chunk<TA, TB, false, NT, TBN>(g, A, B, row0, col0, nextc * KC, vload);
    __builtin_amdgcn_sched_barrier(0);  // keep the next chunk's loads ahead of this chunk's chain
    const int64_t kleft = g.k - c * KC;
    vec acc = (kleft >= KC) ? chain_full<TA, TB, V, CF::LDMB, CF::TR>(As[buf], Bs[buf], ai, bi)
                             : chain_part<TA, TB, V, CF::LDMB, CF::TR>(As[buf], Bs[buf], ai, bi, (int)kleft);
    if (more) store_chunk<TA, TB, NT, TBN, CF::TR>(As[buf ^ 1], Bs[buf ^ 1], nxt);
    __syncthreads();
    buf ^= 1;
    return acc;
  };
  // fast chunk: this and the next chunk full and real (unchecked 16-byte loads)
  auto run_fast = [&](int64_t c) -> vec {
    Raw nxt = load_chunk<TA, TB, true, NT, TBN>(g, A, B, row0, col0, (c + 1) * KC, vload);
    __builtin_amdgcn_sched_barrier(0);  // keep the next chunk's loads ahead of this chunk's chain
    vec acc = chain_full<TA, TB, V, CF::LDMB, CF::TR>(As[buf], Bs[buf], ai, bi);
    __builtin_amdgcn_sched_barrier(0);
    store_chunk<TA, TB, NT, TBN, CF::TR>(As[buf ^ 1], Bs[buf ^ 1], nxt);
    __syncthreads();
    buf ^= 1;
    return acc;
  };
  // the next real chunk after real chunk c of the segment starting at chunk base
  auto next_real = [&](int64_t c, int64_t base) -> int64_t {
    if (!CZ) return c + 1 < nc ? c + 1 : -1;
    if (c + 1 - base < le) return c + 1;
    return (base + spc < nc && lb < le) ? base + spc + lb : -1;
  };
  // a chunk of a group in the segment at base: real chunks run, skipped ones are +0 partials
  auto part = [&](int64_t c, int64_t base) -> vec {
    return (!CZ || (c - base >= lb && c - base < le)) ? run_chunk(c, next_real(c, base)) : zero;
  };

  // Groups of four chunks.  A complete group's partial ((p0 + p1) + (p2 + p3)) is exactly the level-2
  // entry that four pushes would build; it is pushed at level 2 with the group index.  The last group may
  // be partial (nc not a multiple of 4, one segment only): its r chunks form the lowest entries of the
  // final stack (r = 1: p0; 2: p0 + p1; 3: levels 1 and 0 hold p0 + p1 and p2) and start the Result.
  // With segments, spc is a multiple of 4, so a group never spans two.
  const int64_t ng_full = nc >> 2;
  const int64_t gps = nseg > 1 ? spc >> 2 : ng_full + 1;  // groups per segment
  int64_t gj = lb >> 2;
  for (; gj < ng_full; ++gj) {
    const int64_t sgi = nseg > 1 ? gj / gps : 0;
    const int64_t base = sgi * spc;
    const int64_t c = gj * 4, cl = c - base;
    if (CZ && nseg == 1 && cl >= le) break;  // the rest are skipped chunks
    vec qa, qb;  // the group's partial is qa + qb
    if (CZ && (cl + 4 <= lb || cl >= le)) {
      qa = zero;  // a group of skipped chunks: +0 + +0
      qb = zero;
    } else if (tile_in && (!CZ || (cl >= lb && cl + 5 <= le)) && c + 5 <= kfull) {
      vec p0 = run_fast(c);
      vec p1 = run_fast(c + 1);
      qa = p0 + p1;
      vec p2 = run_fast(c + 2);
      vec p3 = run_fast(c + 3);
      qb = p2 + p3;
    } else {
      vec p0 = part(c, base);
      vec p1 = part(c + 1, base);
      qa = p0 + p1;
      vec p2 = part(c + 2, base);
      vec p3 = part(c + 3, base);
      qb = p2 + p3;
    }
    // the 16x16 shapes form the pushed sum at its level (1-5% faster on the weight gradients); the 32x32 shape
    // was 0-1% faster pushing the formed sum
    if (V == 16) S.push_sum(qa, qb, gj, Smem);
    else S.push(qa + qb, gj, Smem);
  }
  // complete groups made only of skipped trailing chunks: their partial is +0
  for (; gj < ng_full; ++gj) S.push(zero + zero, gj, Smem);

  vec r = zero;
  bool have = false;
  const int rem = (int)(nc & 3);
  if (rem) {
    const int64_t c = ng_full * 4;
    vec p0 = part(c, 0);
    if (rem == 1) {
      r = p0;
    } else {
      vec p1 = part(c + 1, 0);
      r = p0 + p1;
      if (rem == 3) r = r + part(c + 2, 0);
    }
    have = true;
  }
  S.result(r, have, ng_full, Smem);

  // store: register v of lane l -> row Mfma::orow, column Mfma::ocol of the wavefront's block
  const int64_t crow0 = row0 + wr * WR, ccol0 = col0 + wc * 64;
  if (g.epi == EPI_DS) {
    uint16_t* C = (uint16_t*)g.c + z1 * g.sc1 + z2 * g.sc2;
    const uint16_t* P = g.ds_p + z1 * g.ds_sp1 + z2 * g.ds_sp2;
    const float* Dv = g.ds_d + z1 * g.ds_sd1 + z2 * g.ds_sd2;
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int64_t i = crow0 + Mfma<V>::orow(v, lane);
      const int64_t j = ccol0 + Mfma<V>::ocol(v, lane);
      if (i < g.m && j < g.n) {
        uint16_t o = 0;
        if (j <= i && (g.ds_window == 0 || j > i - g.ds_window)) {
          const float t = r[v] - Dv[i];
          const float u = bf16_to_f32(P[i * g.ds_ldp + j]) * t;
          o = f32_to_bf16(u * g.ds_scale);
        }
        C[i * g.ldc + j] = o;
      }
    }
    return;
  }
  if (g.epi == EPI_RES) {  // the residual addition RN(res + d) into the fp32 C
    float* C = (float*)g.c + z1 * g.sc1 + z2 * g.sc2;
    const float* R = g.res + z1 * g.sc1 + z2 * g.sc2;
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int64_t i = crow0 + Mfma<V>::orow(v, lane);
      const int64_t j = ccol0 + Mfma<V>::ocol(v, lane);
      if (i < g.m && j < g.n) C[i * g.ldc + j] = R[i * g.ldres + j] + r[v];
    }
    return;
  }
  if (g.epi == EPI_ACCUM) {  // the plan's microbatch accumulation g = RN(g + RN(d * s)) into the fp32 C
    float* C = (float*)g.c + z1 * g.sc1 + z2 * g.sc2;
#pragma unroll
    for (int v = 0; v < V; ++v) {
      const int64_t i = crow0 + Mfma<V>::orow(v, lane);
      const int64_t j = ccol0 + Mfma<V>::ocol(v, lane);
      if (i < g.m && j < g.n) {
        const float t = r[v] * g.epi_scale;
        C[i * g.ldc + j] = C[i * g.ldc + j] + t;
      }
    }
    return;
  }
#pragma unroll
  for (int v = 0; v < V; ++v) {
    const int64_t i = crow0 + Mfma<V>::orow(v, lane);
    const int64_t j = ccol0 + Mfma<V>::ocol(v, lane);
    if (i < g.m && j < g.n) {
      if (g.out_bf16) {
        uint16_t* C = (uint16_t*)g.c + z1 * g.sc1 + z2 * g.sc2;
        C[i * g.ldc + j] = f32_to_bf16(r[v]);
      } else {
        float* C = (float*)g.c + z1 * g.sc1 + z2 * g.sc2;
        C[i * g.ldc + j] = r[v];
      }
    }
  }
}

// Short contractions: at most four chunks (K <= 128: the attention score and dP products), both operands
// k-contiguous and no causal chunk ranges.  One tile is then too little work to hide a workgroup's start
// (launch, first loads) and end (the epilogue's loads and stores), so a persistent grid of two workgroups per
// CU walks the tiles of the batch matrices, each workgroup every G-th tile of its sequence.  The first chunk
// of the next tile is loaded during the last chunk of the current one and its second chunk before the
// current tile's stores (so that waiting for those loads does not wait for the stores); the dS epilogue's P
// and D operands are fetched one chunk before the last.  Per output tile the arithmetic is that of
// gemm_mfma_kernel: chunk chains from +0, then the fold of the at most four partials (two: p0 + p1;
// three: (p0 + p1) + p2; four: (p0 + p1) + (p2 + p3)).
struct ShortTile {
  const uint16_t* A;
  const uint16_t* B;
  int64_t z1, z2, row0, col0;
  bool whole;  // the whole tile inside the m x n matrix
};

// Position in a workgroup's tile sequence: batch matrix z = zl * X + x (X = kXcds when the batch splits evenly
// over the XCDs, else 1; x = the workgroup's XCD), tile row tm, tile column tn; advanced by the number of
// workgroups per XCD group with carries instead of divisions.
constexpr uint32_t kXcds = 8;
struct TileWalk {
  uint32_t zl, tm, tn;
};
// Position in a workgroup's sequence of computed tiles only: matrix zl as above, tile row tm, and the q-th
// tile with a visible entry in that row.
struct LiveWalk {
  uint32_t zl, tm, q;
};

template <bool TA, bool TB, int NC>
__global__ __launch_bounds__(256, 2) void gemm_short_kernel(GemmArgs g) {
  __shared__ __attribute__((aligned(16))) float As[2][A_FLOATS];
  __shared__ __attribute__((aligned(16))) float Bs[2][B_FLOATS];
  // the launcher keeps the tile counts below 2^31
  const uint32_t tiles_n = (uint32_t)((g.n + BN - 1) / BN), tiles_m = (uint32_t)((g.m + BM - 1) / BM);
  const uint32_t per = tiles_m * tiles_n, nb2 = (uint32_t)g.nb2, batch = (uint32_t)g.batch;
  // Workgroup b runs on XCD b % 8 (the dispatcher deals workgroups to the XCDs in turn).  With the batch a
  // multiple of 8 (and the grid too), the workgroups of one XCD take the matrices z = x, x + 8, ...: each
  // XCD's L2 then holds the operands of its own matrices only.
  const uint32_t X = (batch % kXcds == 0 && gridDim.x % kXcds == 0) ? kXcds : 1;
  const uint32_t x = blockIdx.x % X, G = gridDim.x / X, nzl = batch / X;
  const uint32_t step_n = G % tiles_n, step_m = (G / tiles_n) % tiles_m, step_z = G / per;
  const bool ds = g.epi == EPI_DS;
  const int lane = threadIdx.x & 63;
  const int w = threadIdx.x >> 6;
  const int wr = w >> 1, wc = w & 1;
  const int ai = wr * 32 + (lane & 31), bi = wc * 64 + lane;
  // register v, lane l -> block v/16, row (v%4) + 4*(l/32) + 8*((v%16)/4), column l%32: the tile offset of
  // register v is a lane part plus a part common to all lanes (kept in scalar registers; the launcher keeps
  // 64 rows of C and P within 32-bit offsets)
  const int lrow = wr * 32 + 4 * (lane >> 5), lcol = wc * 64 + (lane & 31);
  const uint32_t loff_c = (uint32_t)(lrow * g.ldc + lcol);
  const uint32_t loff_p = (uint32_t)(lrow * g.ds_ldp + lcol);
  auto urow = [](int v) { return (v & 3) + 8 * ((v & 15) >> 2); };
  auto ucol = [](int v) { return 32 * (v >> 4); };
  auto visible = [&](int64_t i, int64_t j) -> bool { return j <= i && (g.ds_window == 0 || j > i - g.ds_window); };

  auto start = [&]() {
    TileWalk W;
    const uint32_t u = blockIdx.x / X, r = u % per;
    W.zl = u / per;
    W.tm = r / tiles_n;
    W.tn = r - W.tm * tiles_n;
    return W;
  };
  auto advance = [&](TileWalk& W) {
    W.tn += step_n;
    uint32_t carry = 0;
    if (W.tn >= tiles_n) { W.tn -= tiles_n; carry = 1; }
    W.tm += step_m + carry;
    carry = 0;
    if (W.tm >= tiles_m) { W.tm -= tiles_m; carry = 1; }
    W.zl += step_z + carry;
  };
  auto done = [&](const TileWalk& W) { return W.zl >= nzl; };
  auto tile_of = [&](const TileWalk& W) -> ShortTile {
    ShortTile T;
    const uint32_t z = W.zl * X + x;
    T.z1 = z / nb2;
    T.z2 = z - (uint32_t)T.z1 * nb2;
    T.row0 = (int64_t)W.tm * BM;
    T.col0 = (int64_t)W.tn * BN;
    T.A = g.a + T.z1 * g.sa1 + T.z2 * g.sa2;
    T.B = g.b + T.z1 * g.sb1 + (g.b_group > 1 ? T.z2 / g.b_group : T.z2) * g.sb2;
    T.whole = T.row0 + BM <= g.m && T.col0 + BN <= g.n;
    return T;
  };
  auto upper_dead = [&](const TileWalk& W) { return g.tri_lower && (int64_t)W.tn * BN > (int64_t)W.tm * BM + BM - 1; };
  auto band_dead = [&](const TileWalk& W) {
    return g.tri_lower && g.kwin > 0 && (int64_t)W.tn * BN + BN - 1 <= (int64_t)W.tm * BM - g.kwin;
  };
  auto band_far = [&](const TileWalk& W) {  // left of the window band and out of every reader's reach
    return band_dead(W) && !g.zero_dead &&
           (int64_t)W.tn * BN + BN - 1 < (int64_t)W.tm * BM - g.kwin - kAttnLead;
  };
  auto in_range = [&](const ShortTile& T, int v) {
    return T.row0 + lrow + urow(v) < g.m && T.col0 + lcol + ucol(v) < g.n;
  };
  // first, the tiles without a visible entry whose +0 the dS epilogue writes
  if (ds && g.tri_lower && (g.zero_dead || g.kwin > 0)) {
    for (TileWalk W = start(); !done(W); advance(W)) {
      if (!((upper_dead(W) && g.zero_dead) || (band_dead(W) && !band_far(W)))) continue;
      const ShortTile T = tile_of(W);
      uint16_t* C = (uint16_t*)g.c + T.z1 * g.sc1 + T.z2 * g.sc2 + T.row0 * g.ldc + T.col0;
#pragma unroll
      for (int v = 0; v < 32; ++v)
        if (in_range(T, v)) (C + urow(v) * g.ldc + ucol(v))[loff_c] = 0;
    }
  }
  // The computed tiles of tile row tm are the columns [row_lo(tm), row_lo(tm) + row_cnt(tm)): below the
  // diagonal tile (tri_lower) and right of the window band.  The workgroups of an XCD group deal out the
  // computed tiles of their matrices (not all tiles), so each gets the same number to within one.
  auto row_lo = [&](uint32_t tm) -> uint32_t {
    if (!g.tri_lower || g.kwin <= 0) return 0;
    const int64_t bound = (int64_t)tm * BM - g.kwin - BN + 1;  // a column tile is computed iff tn * BN > bound
    return bound < 0 ? 0u : (uint32_t)(bound / BN + 1);
  };
  auto row_cnt = [&](uint32_t tm) -> uint32_t {
    uint32_t hi = tiles_n;  // one past the last computed column tile
    if (g.tri_lower) {
      const int64_t h = ((int64_t)tm * BM + BM - 1) / BN + 1;
      if (h < (int64_t)hi) hi = (uint32_t)h;
    }
    const uint32_t lo = row_lo(tm);
    return hi > lo ? hi - lo : 0u;
  };
  uint32_t live = per;  // computed tiles per matrix
  if (g.tri_lower) {
    live = 0;
    for (uint32_t tm = 0; tm < tiles_m; ++tm) live += row_cnt(tm);
  }
  // move forward by n computed tiles (any n)
  auto lmove = [&](LiveWalk& W, uint32_t n) {
    W.zl += n / live;
    W.q += n % live;
    if (!g.tri_lower) {
      W.tm += W.q / tiles_n;
      W.q %= tiles_n;
      W.zl += W.tm / tiles_m;
      W.tm %= tiles_m;
      return;
    }
    for (uint32_t c = row_cnt(W.tm); W.q >= c; c = row_cnt(W.tm)) {
      W.q -= c;
      if (++W.tm == tiles_m) { W.tm = 0; ++W.zl; }
    }
  };
  auto ltile = [&](const LiveWalk& W) {
    TileWalk T;
    T.zl = W.zl;
    T.tm = W.tm;
    T.tn = row_lo(W.tm) + W.q;
    return tile_of(T);
  };
  auto load = [&](const ShortTile& T, int c) -> Raw {
    if (g.vec && T.whole && (int64_t)(c + 1) * KC <= g.k)
      return load_chunk<TA, TB, true, 256, BN>(g, T.A, T.B, T.row0, T.col0, (int64_t)c * KC, true);
    return load_chunk<TA, TB, false, 256, BN>(g, T.A, T.B, T.row0, T.col0, (int64_t)c * KC, g.vec != 0);
  };

  if (live == 0) return;
  LiveWalk cw = {0u, 0u, 0u};
  lmove(cw, blockIdx.x / X);
  if (cw.zl >= nzl) return;
  ShortTile cur = ltile(cw);
  int buf = 0;
  store_chunk<TA, TB, 256, BN>(As[0], Bs[0], load(cur, 0));
  __syncthreads();
  Raw pre;  // chunk 1 of the current tile when its loads went ahead of the previous tile's stores
  bool have_pre = false;
  constexpr int PC = NC >= 2 ? NC - 2 : 0;  // the chunk during which the dS operands are fetched
  for (;;) {
    LiveWalk nw = cw;
    lmove(nw, G);
    const bool has_next = nw.zl < nzl;
    const ShortTile nxt = has_next ? ltile(nw) : cur;
    uint16_t pv[32];
    float dv[16];
    v32f r, p2;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const bool last = c + 1 == NC;
      const bool more = !last || has_next;
      Raw nx;
      if (more) {
        if (last) nx = load(nxt, 0);
        else if (c == 0 && have_pre) nx = pre;
        else nx = load(cur, c + 1);
      }
      if (ds && c == PC) {  // the dS epilogue's operands of this tile (out-of-range entries: +0, not read)
        const uint16_t* P = g.ds_p + cur.z1 * g.ds_sp1 + cur.z2 * g.ds_sp2 + cur.row0 * g.ds_ldp + cur.col0;
        const float* Dv = g.ds_d + cur.z1 * g.ds_sd1 + cur.z2 * g.ds_sd2 + cur.row0 + lrow;
#pragma unroll
        for (int v = 0; v < 32; ++v)
          pv[v] = (cur.whole || in_range(cur, v)) ? (P + urow(v) * g.ds_ldp + ucol(v))[loff_p] : (uint16_t)0;
#pragma unroll
        for (int v = 0; v < 16; ++v) dv[v] = (cur.whole || cur.row0 + lrow + urow(v) < g.m) ? Dv[urow(v)] : 0.0f;
      }
      __builtin_amdgcn_sched_barrier(0);  // keep the loads ahead of this chunk's chain
      const int64_t kleft = g.k - (int64_t)c * KC;
      const v32f acc = kleft >= KC ? chain_full<TA, TB, 32, LDMB>(As[buf], Bs[buf], ai, bi)
                                   : chain_part<TA, TB, 32, LDMB>(As[buf], Bs[buf], ai, bi, (int)kleft);
      __builtin_amdgcn_sched_barrier(0);
      if (more) store_chunk<TA, TB, 256, BN>(As[buf ^ 1], Bs[buf ^ 1], nx);
      __syncthreads();
      buf ^= 1;
      if (c == 0) r = acc;
      else if (c == 1) r = r + acc;
      else if (c == 2) { if (NC == 3) r = r + acc; else p2 = acc; }
      else r = r + (p2 + acc);
    }
    // the next tile's chunk 1 is loaded before this tile's stores, so that waiting for it does not wait for them
    have_pre = NC > 1 && has_next;
    if (have_pre) pre = load(nxt, 1);
    const int64_t off = cur.z1 * g.sc1 + cur.z2 * g.sc2 + cur.row0 * g.ldc + cur.col0;
    if (ds) {
      uint16_t* C = (uint16_t*)g.c + off;
      const int64_t i0 = cur.row0 + lrow, j0 = cur.col0 + lcol;
#pragma unroll
      for (int v = 0; v < 32; ++v) {
        const float d = r[v] - dv[v & 15];
        const float u = bf16_to_f32(pv[v]) * d;
        const uint16_t val = f32_to_bf16(u * g.ds_scale);
        const uint16_t o = visible(i0 + urow(v), j0 + ucol(v)) ? val : (uint16_t)0;
        if (cur.whole || in_range(cur, v)) (C + urow(v) * g.ldc + ucol(v))[loff_c] = o;
      }
    } else if (g.out_bf16) {
      uint16_t* C = (uint16_t*)g.c + off;
#pragma unroll
      for (int v = 0; v < 32; ++v)
        if (cur.whole || in_range(cur, v)) (C + urow(v) * g.ldc + ucol(v))[loff_c] = f32_to_bf16(r[v]);
    } else {
      float* C = (float*)g.c + off;
#pragma unroll
      for (int v = 0; v < 32; ++v)
        if (cur.whole || in_range(cur, v)) (C + urow(v) * g.ldc + ucol(v))[loff_c] = r[v];
    }
    if (!has_next) break;
    cw = nw;
    cur = nxt;
  }
}

// g: A [m][k] and B [n][k] (both k-contiguous), 1 <= chunks <= 4
static hipError_t launch_short(const GemmArgs& g, int64_t nc, int64_t tiles, hipStream_t s) {
  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  int64_t want = 2 * (int64_t)(cus > 0 ? cus : 1);  // two resident workgroups per CU
  if (want >= 8) want -= want % 8;                  // whole groups of the 8 XCDs
  const dim3 grid((unsigned)(tiles < want ? tiles : want));
  if (nc == 1) hipLaunchKernelGGL((gemm_short_kernel<false, true, 1>), grid, dim3(256), 0, s, g);
  else if (nc == 2) hipLaunchKernelGGL((gemm_short_kernel<false, true, 2>), grid, dim3(256), 0, s, g);
  else if (nc == 3) hipLaunchKernelGGL((gemm_short_kernel<false, true, 3>), grid, dim3(256), 0, s, g);
  else hipLaunchKernelGGL((gemm_short_kernel<false, true, 4>), grid, dim3(256), 0, s, g);
  return hipGetLastError();
}

// Workgroup shapes of the general kernel (timed at the 1B shapes; bit-identical results with any of them).
// * Both operands k-contiguous (every forward projection, the head): 64 x 64 tiles with the 16x16 instruction,
//   three workgroups per CU (three wavefronts per SIMD in 168 registers), four fold levels in registers; 3-7%
//   faster than 64 x 128 tiles of the 32x32 instruction with two workgroups per CU.
// * A k-major (weight-gradient layouts): the same 64 x 64 shape with A transposed while staged (LROWX) and
//   three register fold levels, 0-3% faster than the 32x32 shape; left k-major, its 4-byte LDS reads per
//   product (twice as many as with the 32x32 instruction) made it 2-18% slower.
// * Only B k-major (input gradients): 64 x 128 tiles of the 32x32 instruction, two per CU; the transposed
//   16x16 shape was 0-6% slower there.
typedef GemmCfg<16, 1, 3, 4, 4> CfgRowRow;
typedef GemmCfg<16, 1, 3, 4, 3, true> CfgAKMajor;
typedef GemmCfg<32, 2, 2, 3, 2> CfgBKMajor;

template <class CF>
static dim3 general_grid(const GemmArgs& g) {
  return dim3((unsigned)(((g.m + BM - 1) / BM) * ((g.n + CF::TBN - 1) / CF::TBN)), 1, (unsigned)g.batch);
}

template <int MAXL>
static hipError_t launch_maxl(const GemmArgs& g, hipStream_t s) {
  typedef CfgRowRow R;
  typedef CfgAKMajor A;
  typedef CfgBKMajor B;
  if (g.kmode != KMODE_FULL || g.kseg > 0 || g.tri_lower) {  // the causal instantiations
    if (!g.trans_a && g.trans_b)
      hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, false, true, R, true>), general_grid<R>(g), dim3(R::NT), 0, s, g);
    else if (!g.trans_a && !g.trans_b)
      hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, false, false, B, true>), general_grid<B>(g), dim3(B::NT), 0, s, g);
    else if (g.trans_a && !g.trans_b)
      hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, true, false, A, true>), general_grid<A>(g), dim3(A::NT), 0, s, g);
    else
      hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, true, true, A, true>), general_grid<A>(g), dim3(A::NT), 0, s, g);
    return hipGetLastError();
  }
  if (!g.trans_a && g.trans_b)
    hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, false, true, R, false>), general_grid<R>(g), dim3(R::NT), 0, s, g);
  else if (!g.trans_a && !g.trans_b)
    hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, false, false, B, false>), general_grid<B>(g), dim3(B::NT), 0, s, g);
  else if (g.trans_a && !g.trans_b)
    hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, true, false, A, false>), general_grid<A>(g), dim3(A::NT), 0, s, g);
  else
    hipLaunchKernelGGL((gemm_mfma_kernel<MAXL, true, true, A, false>), general_grid<A>(g), dim3(A::NT), 0, s, g);
  return hipGetLastError();
}

int gemm_max_levels() { return 12; }

static bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

hipError_t gemm_launch(const GemmArgs& gin, hipStream_t s) {
  if (gin.m == 0 || gin.n == 0 || gin.batch == 0) return hipSuccess;
  GemmArgs g = gin;
  // 16-byte vector loads need every row start and batch offset on a 16-byte boundary
  g.vec = aligned16(g.a) && aligned16(g.b) && g.lda % 8 == 0 && g.ldb % 8 == 0 && g.sa1 % 8 == 0 &&
          g.sa2 % 8 == 0 && g.sb1 % 8 == 0 && g.sb2 % 8 == 0;
  const int64_t nc = (g.k + KC - 1) / KC;
  int bits = 0;
  while ((int64_t(1) << bits) <= nc) ++bits;  // nc < 2^bits: a push never runs past the top level
  const int64_t tiles = ((g.m + BM - 1) / BM) * ((g.n + BN - 1) / BN);  // short kernel's tiles
  if (!g.trans_a && g.trans_b && nc >= 1 && nc <= 4 && g.kmode == KMODE_FULL && g.kseg == 0 && g.epi != EPI_ACCUM &&
      g.epi != EPI_RES &&
      BM * g.ldc < (int64_t(1) << 31) && BM * g.ds_ldp < (int64_t(1) << 31) && tiles * g.batch < (int64_t(1) << 31) &&
      g.nb2 > 0 && g.batch % g.nb2 == 0)
    return launch_short(g, nc, tiles * g.batch, s);
  if (bits <= 3) return launch_maxl<3>(g, s);
  if (bits <= 5) return launch_maxl<5>(g, s);
  if (bits <= 7) return launch_maxl<7>(g, s);
  if (bits <= 9) return launch_maxl<9>(g, s);
  if (bits <= 11) return launch_maxl<11>(g, s);
  if (bits <= 12) return launch_maxl<12>(g, s);
  return hipErrorInvalidValue;
}

}  // namespace canon
