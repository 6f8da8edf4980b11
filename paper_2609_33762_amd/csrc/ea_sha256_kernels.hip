// Chained prefix-block keys with SHA-256 (FIPS 180-4) on gfx950.
//
// key_i = SHA-256(LE32 tokens of block i || key_{i-1}).  With b a multiple
// of 16 the message is 4b token bytes (b/16 whole 64-byte blocks) followed
// by one final 64-byte block holding key_{i-1}, the 0x80 pad byte and the
// bit length.  The token blocks do not depend on the chain, so the work
// splits in two kernels:
//   sha256_midstates: one lane per key, compresses the b/16 token blocks
//                     from the initial hash value (fully parallel);
//   sha256_chain:     one lane per sequence, runs the final compression of
//                     each key in order, feeding key_{i-1} in as message
//                     words 0..7 (the serial part: one compression per key).
// A lone chain runs at the issue rate of one wave, so the instruction count
// per compression is what matters: rotations are v_alignbit_b32, every
// three-input XOR and Ch/Maj one v_bitop3_b32 (gfx950's three-input logic
// op), sums v_add3_u32; everything stays in VGPRs (no LDS, no scratch).
#include <hip/hip_runtime.h>

#include "ea_internal.hpp"

namespace ea {
namespace {

// FIPS 180-4 section 4.2.2 round constants and section 5.3.3 initial value.
__device__ constexpr uint32_t kRound[64] = {
    0x428a2f98u, 0x71374491u, 0xb5c0fbcfu, 0xe9b5dba5u, 0x3956c25bu, 0x59f111f1u,
    0x923f82a4u, 0xab1c5ed5u, 0xd807aa98u, 0x12835b01u, 0x243185beu, 0x550c7dc3u,
    0x72be5d74u, 0x80deb1feu, 0x9bdc06a7u, 0xc19bf174u, 0xe49b69c1u, 0xefbe4786u,
    0x0fc19dc6u, 0x240ca1ccu, 0x2de92c6fu, 0x4a7484aau, 0x5cb0a9dcu, 0x76f988dau,
    0x983e5152u, 0xa831c66du, 0xb00327c8u, 0xbf597fc7u, 0xc6e00bf3u, 0xd5a79147u,
    0x06ca6351u, 0x14292967u, 0x27b70a85u, 0x2e1b2138u, 0x4d2c6dfcu, 0x53380d13u,
    0x650a7354u, 0x766a0abbu, 0x81c2c92eu, 0x92722c85u, 0xa2bfe8a1u, 0xa81a664bu,
    0xc24b8b70u, 0xc76c51a3u, 0xd192e819u, 0xd6990624u, 0xf40e3585u, 0x106aa070u,
    0x19a4c116u, 0x1e376c08u, 0x2748774cu, 0x34b0bcb5u, 0x391c0cb3u, 0x4ed8aa4au,
    0x5b9cca4fu, 0x682e6ff3u, 0x748f82eeu, 0x78a5636fu, 0x84c87814u, 0x8cc70208u,
    0x90befffau, 0xa4506cebu, 0xbef9a3f7u, 0xc67178f2u};

__device__ constexpr uint32_t kInit[8] = {0x6a09e667u, 0xbb67ae85u, 0x3c6ef372u,
                                          0xa54ff53au, 0x510e527fu, 0x9b05688cu,
                                          0x1f83d9abu, 0x5be0cd19u};

__device__ __forceinline__ uint32_t rotr(uint32_t x, int n) {
  return __builtin_amdgcn_alignbit(x, x, n);
}

// v_bitop3_b32 truth tables over inputs (x, y, z) = (0xF0, 0xCC, 0xAA).
constexpr uint32_t kXor3 = 0x96;  // x ^ y ^ z
constexpr uint32_t kCh = 0xCA;    // x ? y : z
constexpr uint32_t kMaj = 0xE8;   // majority

template <uint32_t TABLE>
__device__ __forceinline__ uint32_t bitop3(uint32_t x, uint32_t y, uint32_t z) {
  return __builtin_amdgcn_bitop3_b32(x, y, z, TABLE);
}

// One compression: st <- st + rounds(st, w).  w is consumed (used as the
// rolling 16-word message schedule).
__device__ __forceinline__ void compress(uint32_t st[8], uint32_t w[16]) {
  uint32_t a = st[0], b = st[1], c = st[2], d = st[3];
  uint32_t e = st[4], f = st[5], g = st[6], h = st[7];
#pragma unroll
  for (int t = 0; t < 64; ++t) {
    uint32_t wt;
    if (t < 16) {
      wt = w[t];
    } else {
      const uint32_t w2 = w[(t - 2) & 15], w15 = w[(t - 15) & 15];
      const uint32_t s1 = bitop3<kXor3>(rotr(w2, 17), rotr(w2, 19), w2 >> 10);
      const uint32_t s0 = bitop3<kXor3>(rotr(w15, 7), rotr(w15, 18), w15 >> 3);
      wt = s1 + w[(t - 7) & 15] + s0 + w[t & 15];
      w[t & 15] = wt;
    }
    const uint32_t S1 = bitop3<kXor3>(rotr(e, 6), rotr(e, 11), rotr(e, 25));
    const uint32_t ch = bitop3<kCh>(e, f, g);
    const uint32_t t1 = h + S1 + ch + kRound[t] + wt;
    const uint32_t S0 = bitop3<kXor3>(rotr(a, 2), rotr(a, 13), rotr(a, 22));
    const uint32_t mj = bitop3<kMaj>(a, b, c);
    const uint32_t t2 = S0 + mj;
    h = g; g = f; f = e; e = d + t1;
    d = c; c = b; b = a; a = t1 + t2;
  }
  st[0] += a; st[1] += b; st[2] += c; st[3] += d;
  st[4] += e; st[5] += f; st[6] += g; st[7] += h;
}

// index of the sequence owning key g: largest s with key_off[s] <= g
__device__ __forceinline__ int32_t owner(const int64_t *key_off, int32_t n_seqs,
                                         int64_t g) {
  int32_t lo = 0, hi = n_seqs - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (key_off[mid] <= g) lo = mid; else hi = mid - 1;
  }
  return lo;
}

__global__ __launch_bounds__(256) void sha256_midstates(
    const int32_t *__restrict__ tokens, const int64_t *__restrict__ key_off,
    const int64_t *__restrict__ tok_off, int32_t n_seqs, int64_t n_keys,
    int32_t block_tokens, uint32_t *__restrict__ mid) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= n_keys) return;
  const int32_t s = owner(key_off, n_seqs, g);
  const int64_t i = g - key_off[s];
  const int32_t *tok = tokens + tok_off[s] + i * block_tokens;
  uint32_t st[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) st[j] = kInit[j];
  for (int32_t c = 0; c < block_tokens; c += 16) {
    uint32_t w[16];
#pragma unroll
    for (int j = 0; j < 16; ++j)  // LE32 token bytes read as a big-endian word
      w[j] = __builtin_bswap32((uint32_t)tok[c + j]);
    compress(st, w);
  }
  uint4 *out = reinterpret_cast<uint4 *>(mid + 8 * g);
  out[0] = make_uint4(st[0], st[1], st[2], st[3]);
  out[1] = make_uint4(st[4], st[5], st[6], st[7]);
}

__global__ __launch_bounds__(64) void sha256_chain(
    const uint32_t *__restrict__ mid, const int64_t *__restrict__ key_off,
    int32_t n_seqs, uint32_t len_bits, const uint8_t *__restrict__ parents,
    uint8_t *__restrict__ keys) {
  const int32_t s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= n_seqs) return;
  uint32_t prev[8];
  if (parents != nullptr) {
    const uint8_t *p = parents + 32 * (int64_t)s;
#pragma unroll
    for (int j = 0; j < 8; ++j)
      prev[j] = ((uint32_t)p[4 * j] << 24) | ((uint32_t)p[4 * j + 1] << 16) |
                ((uint32_t)p[4 * j + 2] << 8) | (uint32_t)p[4 * j + 3];
  } else {
#pragma unroll
    for (int j = 0; j < 8; ++j) prev[j] = 0;
  }
  const int64_t k0 = key_off[s], k1 = key_off[s + 1];
  if (k0 == k1) return;
  const uint4 *m = reinterpret_cast<const uint4 *>(mid);
  uint4 nx0 = m[2 * k0], nx1 = m[2 * k0 + 1];
  for (int64_t k = k0; k < k1; ++k) {
    uint32_t st[8] = {nx0.x, nx0.y, nx0.z, nx0.w, nx1.x, nx1.y, nx1.z, nx1.w};
    if (k + 1 < k1) {  // the next midstate does not depend on the chain
      nx0 = m[2 * (k + 1)];
      nx1 = m[2 * (k + 1) + 1];
    }
    uint32_t w[16] = {prev[0], prev[1], prev[2], prev[3], prev[4], prev[5],
                      prev[6], prev[7], 0x80000000u, 0u, 0u, 0u, 0u, 0u, 0u,
                      len_bits};
    compress(st, w);
    uint4 *out = reinterpret_cast<uint4 *>(keys + 32 * k);
    out[0] = make_uint4(__builtin_bswap32(st[0]), __builtin_bswap32(st[1]),
                        __builtin_bswap32(st[2]), __builtin_bswap32(st[3]));
    out[1] = make_uint4(__builtin_bswap32(st[4]), __builtin_bswap32(st[5]),
                        __builtin_bswap32(st[6]), __builtin_bswap32(st[7]));
#pragma unroll
    for (int j = 0; j < 8; ++j) prev[j] = st[j];
  }
}

}  // namespace

hipError_t launch_sha256_midstates(const int32_t *d_tokens,
                                   const int64_t *d_key_offsets,
                                   const int64_t *d_tok_offsets, int32_t n_seqs,
                                   int64_t n_keys, int32_t block_tokens,
                                   uint32_t *d_mid, hipStream_t stream) {
  if (n_keys <= 0) return hipSuccess;
  const int64_t blocks = (n_keys + 255) / 256;
  hipLaunchKernelGGL(sha256_midstates, dim3((unsigned)blocks), dim3(256), 0, stream,
                     d_tokens, d_key_offsets, d_tok_offsets, n_seqs, n_keys,
                     block_tokens, d_mid);
  return hipGetLastError();
}

hipError_t launch_sha256_chain(const uint32_t *d_mid,
                               const int64_t *d_key_offsets, int32_t n_seqs,
                               int32_t block_tokens, const uint8_t *d_parents,
                               uint8_t *d_keys, hipStream_t stream) {
  if (n_seqs <= 0) return hipSuccess;
  // message = 4b token bytes + 32 key bytes
  const uint32_t len_bits = (uint32_t)(8u * (4u * (uint32_t)block_tokens + 32u));
  const int blocks = (n_seqs + 63) / 64;
  hipLaunchKernelGGL(sha256_chain, dim3(blocks), dim3(64), 0, stream, d_mid,
                     d_key_offsets, n_seqs, len_bits, d_parents, d_keys);
  return hipGetLastError();
}

}  // namespace ea
