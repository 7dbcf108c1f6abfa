// hash.hip - the canonical state hash H1 on the device.
//
// H1 (this library's definition; the paper hashes every step's state on the host and leaves the function
// open): SHA-256 (FIPS 180-4) over a fixed tree.
//   * a tensor of n bytes is cut into nb = ceil(n/64) blocks of 64 bytes (the last may be shorter) and
//     W = max(1, ceil(nb/1024)) leaves; leaf l holds blocks l, l+W, l+2W, ... in order (interleaved, so the
//     lanes of a wavefront, one leaf each, read neighbouring blocks);
//   * leaf digest = SHA-256(leaf bytes); the leaf digests fold pairwise level by level,
//     SHA-256(left || right), an odd last node passing up unchanged;
//   * tensor digest = SHA-256(0x02 || index as 8 bytes LE || n as 8 bytes LE || root);
//   * state digest = SHA-256(0x03 || tensor digests in order).
// Integer arithmetic only: the result is the same on every device.
#include <hip/hip_runtime.h>

#include "canon_internal.h"

namespace canon {

// SHA-256 round constants and initial state (FIPS 180-4, sections 4.2.2 and 5.3.3)
__constant__ uint32_t kSha256K[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u, 0x923f82a4u, 0xab1c5ed5u,
    0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u, 0x72be5d74u, 0x80deb1feu, 0x9bdc06a7u, 0xc19bf174u,
    0xe49b69c1u, 0xefbe4786u, 0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu, 0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau,
    0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u, 0xc6e00bf3u, 0xd5a79147u, 0x06ca6351u, 0x14292967u,
    0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu, 0x53380d13u, 0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u,
    0xa2bfe8a1u, 0xa81a664bu, 0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u,
    0x19a4c116u, 0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au, 0x5b9cca4fu, 0x682e6ff3u,
    0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u, 0x90befffau, 0xa4506cebu, 0xbef9a3f7u, 0xc67178f2u};
constexpr uint32_t kSha256H0[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u, 0xa54ff53au,
                                   0x510e527fu, 0x9b05688cu, 0x1f83d9abu, 0x5be0cd19u};

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) { return (x >> n) | (x << (32 - n)); }

struct Sha {
  uint32_t h[8];
  __device__ void init() {
#pragma unroll
    for (int i = 0; i < 8; ++i) h[i] = kSha256H0[i];
  }
  // one 64-byte block given as 16 big-endian words
  __device__ void compress(const uint32_t (&m)[16]) {
    uint32_t w[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) w[i] = m[i];
    uint32_t a = h[0], b = h[1], c = h[2], d = h[3], e = h[4], f = h[5], g = h[6], hh = h[7];
#pragma unroll
    for (int t = 0; t < 64; ++t) {
      uint32_t wt;
      if (t < 16) {
        wt = w[t];
      } else {
        const uint32_t w15 = w[(t + 1) & 15], w2 = w[(t + 14) & 15];
        const uint32_t s0 = rotr(w15, 7) ^ rotr(w15, 18) ^ (w15 >> 3);
        const uint32_t s1 = rotr(w2, 17) ^ rotr(w2, 19) ^ (w2 >> 10);
        wt = w[t & 15] + s0 + w[(t + 9) & 15] + s1;
        w[t & 15] = wt;
      }
      const uint32_t S1 = rotr(e, 6) ^ rotr(e, 11) ^ rotr(e, 25);
      const uint32_t ch = (e & f) ^ (~e & g);
      const uint32_t t1 = hh + S1 + ch + kSha256K[t] + wt;
      const uint32_t S0 = rotr(a, 2) ^ rotr(a, 13) ^ rotr(a, 22);
      const uint32_t mj = (a & b) ^ (a & c) ^ (b & c);
      const uint32_t t2 = S0 + mj;
      hh = g; g = f; f = e; e = d + t1; d = c; c = b; b = a; a = t1 + t2;
    }
    h[0] += a; h[1] += b; h[2] += c; h[3] += d; h[4] += e; h[5] += f; h[6] += g; h[7] += hh;
  }
};

// Streaming byte writer for short messages assembled in registers (node, tensor and state digests).
struct ShaStream {
  Sha s;
  uint32_t m[16];
  int fill;        // bytes in the current block
  uint64_t total;  // bytes so far
  __device__ void init() {
    s.init();
    fill = 0;
    total = 0;
#pragma unroll
    for (int i = 0; i < 16; ++i) m[i] = 0;
  }
  __device__ void byte(uint32_t v) {
    m[fill >> 2] |= (v & 0xFFu) << (24 - 8 * (fill & 3));
    ++fill;
    ++total;
    if (fill == 64) {
      s.compress(m);
      fill = 0;
      for (int i = 0; i < 16; ++i) m[i] = 0;
    }
  }
  __device__ void word_be(uint32_t v) {
    byte(v >> 24); byte(v >> 16); byte(v >> 8); byte(v);
  }
  __device__ void finish(uint32_t (&out)[8]) {
    const uint64_t bits = total * 8;
    byte(0x80);
    while (fill != 56) byte(0);
    for (int i = 7; i >= 0; --i) byte((uint32_t)(bits >> (8 * i)));
#pragma unroll
    for (int i = 0; i < 8; ++i) out[i] = s.h[i];
  }
};

__device__ __forceinline__ uint32_t bswap(uint32_t x) { return __builtin_bswap32(x); }

// Leaves of every tensor: one thread per leaf; a workgroup covers up to 256 leaves of one tensor.
__global__ __launch_bounds__(256) void hash_leaves_kernel(const HashTensor* __restrict__ tens,
                                                          const int32_t* __restrict__ wg_tensor,
                                                          const int64_t* __restrict__ wg_first,
                                                          uint32_t* __restrict__ leaf_out) {
  const HashTensor T = tens[wg_tensor[blockIdx.x]];
  const int64_t l = wg_first[blockIdx.x] + threadIdx.x;
  if (l >= T.leaves) return;
  const uint8_t* base = (const uint8_t*)T.ptr;
  const int64_t n = T.nbytes, nb = (n + 63) / 64, W = T.leaves;
  const int64_t nfull = n / 64;  // blocks with all 64 bytes
  Sha s;
  s.init();
  uint64_t len = 0;
  int64_t b = l;
  for (; b < nfull; b += W) {
    uint32_t m[16];
    if (T.aligned) {
      const uint4* p = reinterpret_cast<const uint4*>(base + b * 64);
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const uint4 u = p[q];
        m[4 * q] = bswap(u.x); m[4 * q + 1] = bswap(u.y); m[4 * q + 2] = bswap(u.z); m[4 * q + 3] = bswap(u.w);
      }
    } else {
      for (int i = 0; i < 16; ++i) {
        const uint8_t* q = base + b * 64 + 4 * i;
        m[i] = ((uint32_t)q[0] << 24) | ((uint32_t)q[1] << 16) | ((uint32_t)q[2] << 8) | (uint32_t)q[3];
      }
    }
    s.compress(m);
    len += 64;
  }
  // the partial last block (if this leaf owns it), then the padding
  uint32_t m[16];
  for (int i = 0; i < 16; ++i) m[i] = 0;
  int fill = 0;
  if (b == nfull && nfull < nb) {
    const int tail = (int)(n - nfull * 64);
    for (int i = 0; i < tail; ++i) m[i >> 2] |= (uint32_t)base[nfull * 64 + i] << (24 - 8 * (i & 3));
    fill = tail;
    len += tail;
  }
  m[fill >> 2] |= 0x80u << (24 - 8 * (fill & 3));
  if (fill >= 56) {
    s.compress(m);
    for (int i = 0; i < 16; ++i) m[i] = 0;
  }
  const uint64_t bits = len * 8;
  m[14] = (uint32_t)(bits >> 32);
  m[15] = (uint32_t)bits;
  s.compress(m);
  uint32_t* o = leaf_out + 8 * (T.leaf_offset + l);
#pragma unroll
  for (int i = 0; i < 8; ++i) o[i] = s.h[i];
}

// Pairwise fold of each tensor's leaf digests (one workgroup per tensor, ping-pong between two buffers),
// then the tensor digest.
__global__ __launch_bounds__(256) void hash_tree_kernel(const HashTensor* __restrict__ tens, uint32_t* bufA,
                                                        uint32_t* bufB, uint32_t* __restrict__ tensor_out) {
  const HashTensor T = tens[blockIdx.x];
  uint32_t* src = bufA + 8 * T.leaf_offset;
  uint32_t* dst = bufB + 8 * T.leaf_offset;
  int64_t m = T.leaves;
  while (m > 1) {
    const int64_t pairs = m / 2;
    for (int64_t i = threadIdx.x; i < (m + 1) / 2; i += 256) {
      uint32_t out[8];
      if (i < pairs) {
        Sha s;
        s.init();
        uint32_t blk[16];
#pragma unroll
        for (int k = 0; k < 16; ++k) blk[k] = src[8 * (2 * i) + k];  // left then right, already big-endian words
        s.compress(blk);
        uint32_t pad[16] = {0x80000000u, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 512u};
        s.compress(pad);
#pragma unroll
        for (int k = 0; k < 8; ++k) out[k] = s.h[k];
      } else {  // odd last node passes up
#pragma unroll
        for (int k = 0; k < 8; ++k) out[k] = src[8 * (2 * i) + k];
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) dst[8 * i + k] = out[k];
    }
    __syncthreads();
    uint32_t* t = src;
    src = dst;
    dst = t;
    m = (m + 1) / 2;
  }
  if (threadIdx.x == 0) {
    ShaStream st;
    st.init();
    st.byte(0x02);
    for (int i = 0; i < 8; ++i) st.byte((uint32_t)((uint64_t)blockIdx.x >> (8 * i)));
    for (int i = 0; i < 8; ++i) st.byte((uint32_t)((uint64_t)T.nbytes >> (8 * i)));
    for (int k = 0; k < 8; ++k) st.word_be(src[k]);
    uint32_t d[8];
    st.finish(d);
    for (int k = 0; k < 8; ++k) tensor_out[8 * blockIdx.x + k] = d[k];
  }
}

// state digest = SHA-256(0x03 || tensor digests); written as 32 bytes
__global__ void hash_state_kernel(int64_t n_tensors, const uint32_t* __restrict__ tensor_digests,
                                  uint8_t* __restrict__ out) {
  if (threadIdx.x != 0) return;
  ShaStream st;
  st.init();
  st.byte(0x03);
  for (int64_t t = 0; t < n_tensors; ++t)
    for (int k = 0; k < 8; ++k) st.word_be(tensor_digests[8 * t + k]);
  uint32_t d[8];
  st.finish(d);
  for (int k = 0; k < 8; ++k)
    for (int i = 0; i < 4; ++i) out[4 * k + i] = (uint8_t)(d[k] >> (24 - 8 * i));
}

int64_t hash_leaf_count(int64_t nbytes) {
  const int64_t nb = (nbytes + 63) / 64;
  const int64_t w = (nb + 1023) / 1024;
  return w < 1 ? 1 : w;
}

hipError_t hash_launch(int64_t n_tensors, const HashTensor* tens_dev, int64_t n_wg, const int32_t* wg_tensor,
                       const int64_t* wg_first, uint32_t* leaf_a, uint32_t* leaf_b, uint32_t* tensor_digests,
                       uint8_t* out, hipStream_t s) {
  if (n_wg > 0) hipLaunchKernelGGL(hash_leaves_kernel, dim3((unsigned)n_wg), dim3(256), 0, s, tens_dev, wg_tensor,
                                   wg_first, leaf_a);
  if (n_tensors > 0)
    hipLaunchKernelGGL(hash_tree_kernel, dim3((unsigned)n_tensors), dim3(256), 0, s, tens_dev, leaf_a, leaf_b,
                       tensor_digests);
  hipLaunchKernelGGL(hash_state_kernel, dim3(1), dim3(64), 0, s, n_tensors, tensor_digests, out);
  return hipGetLastError();
}

}  // namespace canon
