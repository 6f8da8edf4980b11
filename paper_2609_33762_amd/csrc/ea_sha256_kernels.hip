// Chained prefix-block keys with SHA-256 (FIPS 180-4) on gfx950.
//
// key_i = SHA-256(LE32 tokens of block i || key_{i-1}).  With b a multiple
// of 16 the message is 4b token bytes (b/16 whole 64-byte blocks) followed
// by one final 64-byte block holding key_{i-1}, the 0x80 pad byte and the
// bit length.  The token blocks do not depend on the chain, so the work
// splits in two kernels:
//   sha256_midstates: one lane per key, compresses the b/16 token blocks
//                     from the initial hash value (fully parallel);
//   sha256_midstates_split: the same for few keys of several blocks, a
//                     workgroup of two waves per four keys (one per
//                     16-lane row), the schedules on the second wave;
//   sha256_chain:     two lanes per sequence, run the final compression of
//                     each key in order, feeding key_{i-1} in as message
//                     words 0..7 (the serial part: one compression per key);
//   sha256_chain_lane: the same with one lane per sequence, for batches of
//                     sequences large enough to give every SIMD more than
//                     one wave of the two-lane form;
//   sha256_chain_split: the same for few long chains, a workgroup of two
//                     waves per four sequences (one per 16-lane row), with
//                     the message schedule moved to the second wave.
// A lone chain runs at the issue rate of one wave, so the instructions per
// compression set its speed: rotations are v_alignbit_b32, every
// three-input XOR and Ch/Maj one v_bitop3_b32 (gfx950's three-input logic
// op), sums v_add3_u32; everything stays in VGPRs (no LDS, no scratch).
// Splitting the working state and the message schedule over two lanes
// (below) brings a chained compression to 1,162 instructions from 1,378 in
// one lane, and gives twice as many waves for a given number of sequences.
// The split costs lane-instructions (2 x 1,162 per key against 1,378), so
// once the two-lane form would stack waves on a SIMD the one-lane form
// finishes first: 65,536 sequences of 16 keys take 47 us in one lane
// against 66 us in two, while 32,768 of 32 keys (one two-lane wave per
// SIMD) take 83 us against 72 us.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <mutex>

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
template <typename Off>
__device__ __forceinline__ int32_t owner(const Off *key_off, int32_t n_seqs, int64_t g) {
  int32_t lo = 0, hi = n_seqs - 1;
  while (lo < hi) {
    const int32_t mid = (lo + hi + 1) >> 1;
    if (key_off[mid] <= g) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// The parent key of sequence s as eight big-endian words (zero without
// parents: the chain starts from the all-zero root).
__device__ __forceinline__ void parent_words(const uint8_t *parents, int32_t s,
                                             uint32_t prev[8]) {
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
}

// Offsets (Off) are 32-bit when every key and token offset fits, which
// halves their upload; 64-bit otherwise.
template <typename Off>
__global__ __launch_bounds__(256) void sha256_midstates(
    const int32_t *__restrict__ tokens, const Off *__restrict__ key_off,
    const Off *__restrict__ tok_off, int32_t n_seqs, int64_t n_keys,
    int32_t block_tokens, uint32_t *__restrict__ mid) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  // n_keys bounds the grid; the offsets hold the keys there are (fewer when
  // the offsets were derived on the device from a bound)
  if (g >= n_keys || g >= (int64_t)key_off[n_seqs]) return;
  const int32_t s = owner(key_off, n_seqs, g);
  const int64_t i = g - (int64_t)key_off[s];
  if (i < 0 || g >= (int64_t)key_off[s + 1]) return;  // offsets not increasing: nothing to do
  const int32_t *tok = tokens + (int64_t)tok_off[s] + i * block_tokens;
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

// Two lanes per sequence: lane 2q holds a..d of sequence q's working
// state, lane 2q+1 holds e..h.  A round is the same instruction stream on
// both lanes with per-lane rotation amounts: Sigma0(a) and Maj(a, b, c) on
// the a-side, Sigma1(e) and Ch(e, f, g) on the e-side (Maj(a, b, c) equals
// Ch(a ^ c, b, c), so one bitop3 serves both); T1 crosses from the e-lane to
// the a-lane and d from the a-lane to the e-lane through DPP lane moves.
// The message schedule is split the same way: one step computes W_2j on
// the e-lane and W_2j+1 on the a-lane, each lane taking the two terms that
// live on the other lane through a lane swap.
constexpr int kPermFromE = 0xF5;  // quad_perm [1,1,3,3]: read lane 2q+1
constexpr int kPermFromA = 0xA0;  // quad_perm [0,0,2,2]: read lane 2q
constexpr int kPermSwap = 0xB1;   // quad_perm [1,0,3,2]: read the other lane
constexpr uint32_t kXorAnd = 0x78;  // x ^ (y & z)

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_from(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}

template <typename Off>
__global__ __launch_bounds__(64) void sha256_chain(
    const uint32_t *__restrict__ mid, const Off *__restrict__ key_off,
    int32_t n_seqs, uint32_t len_bits, const uint8_t *__restrict__ parents,
    uint8_t *__restrict__ keys) {
  const int lane = threadIdx.x;
  const bool e_side = lane & 1;
  const int32_t s = blockIdx.x * 32 + (lane >> 1);
  if (s >= n_seqs) return;  // both lanes of a pair leave together
  const uint32_t r1c = e_side ? 6 : 2, r2c = e_side ? 11 : 13, r3c = e_side ? 25 : 22;
  const uint32_t m = e_side ? 0u : 0xffffffffu;
  uint32_t prev[8];
  parent_words(parents, s, prev);
  const int64_t k0 = key_off[s], k1 = key_off[s + 1];
  const uint4 *mh = reinterpret_cast<const uint4 *>(mid);
  uint4 nx = k0 < k1 ? mh[2 * k0 + (e_side ? 1 : 0)] : make_uint4(0, 0, 0, 0);
  // Take the first midstate before the loop.  Memory operations complete in
  // issue order as far as the wait counter is concerned, so a load still
  // pending at the loop head would make every key wait for the previous
  // key's store to be acknowledged; with none pending there, a key waits
  // only for the prefetch of its midstate, issued a whole compression
  // earlier and ahead of that store.
  asm volatile("" ::"v"(nx.x), "v"(nx.y), "v"(nx.z), "v"(nx.w));
  // message words in pairs: x[j] holds W_2j on the e-lane, W_2j+1 on the
  // a-lane; x[0..3] come from the previous key, x[4..7] are the padding
  const uint32_t pad8 = e_side ? 0x80000000u : 0u;   // (W8, W9)
  const uint32_t pad14 = e_side ? 0u : len_bits;      // (W14, W15)
  uint32_t x[8];
  {
    // the parent key: e-lane (W_2j), a-lane (W_2j+1)
    x[0] = e_side ? prev[0] : prev[1];
    x[1] = e_side ? prev[2] : prev[3];
    x[2] = e_side ? prev[4] : prev[5];
    x[3] = e_side ? prev[6] : prev[7];
  }
  for (int64_t k = k0; k < k1; ++k) {
    const uint4 h0 = nx;  // this lane's half of the midstate
    if (k + 1 < k1) nx = mh[2 * (k + 1) + (e_side ? 1 : 0)];
    uint32_t s0 = h0.x, s1 = h0.y, s2 = h0.z, s3 = h0.w;
    uint32_t X[32];
    X[0] = x[0]; X[1] = x[1]; X[2] = x[2]; X[3] = x[3];
    X[4] = pad8; X[5] = 0u; X[6] = 0u; X[7] = pad14;
#pragma unroll
    for (int t = 0; t < 64; ++t) {
      const int j = t >> 1;
      if ((t & 1) == 0 && j >= 8) {
        // W_2j (e-lane) and W_2j+1 (a-lane) at once: the partner's terms
        // come through a lane swap of a register each lane fills for it
        const uint32_t r1 = e_side ? X[j - 3] : X[j - 4];
        const uint32_t r2 = e_side ? X[j - 7] : X[j - 8];
        const uint32_t x1 = X[j - 1];
        const uint32_t g1 = bitop3<kXor3>(rotr(x1, 17), rotr(x1, 19), x1 >> 10);
        const uint32_t g0 = bitop3<kXor3>(rotr(r2, 7), rotr(r2, 18), r2 >> 3);
        X[j] = (g1 + dpp_from<kPermSwap>(g0)) + (X[j - 8] + dpp_from<kPermSwap>(r1));
      }
      // W_t on the e-lane: its own word for even t, the a-lane's for odd t
      const uint32_t wt = (t & 1) ? dpp_from<kPermFromA>(X[j]) : X[j];
      const uint32_t S = bitop3<kXor3>(__builtin_amdgcn_alignbit(s0, s0, r1c),
                                       __builtin_amdgcn_alignbit(s0, s0, r2c),
                                       __builtin_amdgcn_alignbit(s0, s0, r3c));
      const uint32_t F = bitop3<kCh>(bitop3<kXorAnd>(s0, s2, m), s1, s2);
      const uint32_t U = S + F;                       // a-lane: T2
      const uint32_t T1 = U + s3 + (kRound[t] + wt);  // e-lane: T1
      // the move runs on every lane (a DPP move cannot sit under a branch)
      const uint32_t dA = dpp_from<kPermFromA>(s3);
      const uint32_t Q = e_side ? dA : U;
      const uint32_t nw = dpp_from<kPermFromE>(T1) + Q;
      s3 = s2; s2 = s1; s1 = s0; s0 = nw;
    }
    const uint32_t o0 = h0.x + s0, o1 = h0.y + s1, o2 = h0.z + s2, o3 = h0.w + s3;
    uint4 *out = reinterpret_cast<uint4 *>(keys + 32 * k + (e_side ? 16 : 0));
    *out = make_uint4(__builtin_bswap32(o0), __builtin_bswap32(o1), __builtin_bswap32(o2),
                      __builtin_bswap32(o3));
    // the key is the next message's words 0..7 (H0..H3 on the a-lane, H4..H7
    // on the e-lane): x[0] = (H0, H1), x[1] = (H2, H3), x[2] = (H4, H5),
    // x[3] = (H6, H7) as (e-lane, a-lane)
    const uint32_t a0 = dpp_from<kPermFromA>(o0), a2 = dpp_from<kPermFromA>(o2);
    const uint32_t e1 = dpp_from<kPermFromE>(o1), e3 = dpp_from<kPermFromE>(o3);
    x[0] = e_side ? a0 : o1;
    x[1] = e_side ? a2 : o3;
    x[2] = e_side ? o0 : e1;
    x[3] = e_side ? o2 : e3;
  }
}

// One sequence per workgroup of two waves: wave 0 runs the rounds, wave 1
// the message schedule, handed over through LDS.
//
// Rounds wave.  Lanes 0..3 of every row of 16 hold the a-side (a, b, c, d)
// of the working state, lanes 12..15 the e-side (e, f, g, h); lanes 4..11
// compute values nobody reads.  Writing A_t and E_t for the new a and e of
// round t, the round is
//   E_t = Sigma1(E_t-1) + Ch(E_t-1, E_t-2, E_t-3) + (E_t-4 + A_t-4 + K_t + W_t)
//   A_t = E_t + Sigma0(A_t-1) + Maj(A_t-1, A_t-2, A_t-3) - A_t-4
// (T1 = E_t - d, A_t = T1 + T2).  Both lanes run one instruction stream
// with per-lane rotation amounts (Maj(a, b, c) = Ch(a ^ c, b, c), so one
// v_bitop3 serves both sides): G = Sigma + Ch/Maj + V, where V holds the
// bracket on the e-side and -A_t-4 on the a-side, and one DPP add gives
// both lanes their new value: row_shl:12 brings the e-lane's G to the
// a-lane, and the e-lane, whose source lies outside the row, adds zero.
// V for the next round takes two instructions that fill the DPP add's
// wait states: a row_shr:12 add brings A_t-3 to the e-lane (zero to the
// a-lane) plus K + W (1 on the a-lane), then v_xad_u32 adds E_t-3 on the
// e-lane and ~A_t-3 on the a-lane (~x + 1 = -x).  Ten instructions per
// round, no wait states, and every VGPR a DPP instruction reads was
// written at least two instructions before it.  The rounds sit in asm
// blocks of up to four (the compiler adds a wait state between blocks);
// volatile keeps them where they are written relative to the barriers.
//
// Schedule wave.  Lane j of a row holds W_T0-16+j and computes W_T0+j for
// the 16 words of a part: the terms from the previous part in three DPP
// passes, then seven steps in which lane j takes sigma1 of lane j - 2 and
// W_t-7 from lane j - 7 (two steps old, hence no wait states); after step s
// lanes 0 .. 2s + 1 hold final words.
//
// Per key: the rounds wave runs rounds 0..11 from the previous key and the
// fixed padding words while the schedule wave computes words 16..31; a
// barrier; the rounds wave reads them and runs rounds 12..26 while words
// 32..47 are computed; a barrier; rounds 27..42 | words 48..63; a barrier;
// rounds 43..63, the key into LDS; a barrier, after which the schedule
// wave reads the key, stores the previous one and starts the next key's
// words.  Each wave runs its own loop with the same four barriers per key.
#define EA_RND(S0, S1, S2, K, VI, VO, NW)                                                    \
  "v_alignbit_b32 %[r1], %[" S0 "], %[" S0 "], %[c1]\n\t"                                    \
  "v_alignbit_b32 %[r2], %[" S0 "], %[" S0 "], %[c2]\n\t"                                    \
  "v_alignbit_b32 %[r3], %[" S0 "], %[" S0 "], %[c3]\n\t"                                    \
  "v_bitop3_b32 %[x], %[" S0 "], %[" S2 "], %[m] bitop3:0x78\n\t"                            \
  "v_bitop3_b32 %[F], %[x], %[" S1 "], %[" S2 "] bitop3:0xca\n\t"                            \
  "v_bitop3_b32 %[S], %[r1], %[r2], %[r3] bitop3:0x96\n\t"                                   \
  "v_add3_u32 %[G], %[S], %[F], %[" VI "]\n\t"                                               \
  "v_add_u32_dpp %[P], %[" S2 "], %[" K "] row_shr:12 row_mask:0xf bank_mask:0xf "           \
  "bound_ctrl:1\n\t"                                                                         \
  "v_xad_u32 %[" VO "], %[" S2 "], %[m], %[P]\n\t"                                           \
  "v_add_u32_dpp %[" NW "], %[G], %[G] row_shl:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"
// The last round of a compression: no next V, two wait states instead.
#define EA_RND_LAST(S0, S1, S2, VI, NW)                                                      \
  "v_alignbit_b32 %[r1], %[" S0 "], %[" S0 "], %[c1]\n\t"                                    \
  "v_alignbit_b32 %[r2], %[" S0 "], %[" S0 "], %[c2]\n\t"                                    \
  "v_alignbit_b32 %[r3], %[" S0 "], %[" S0 "], %[c3]\n\t"                                    \
  "v_bitop3_b32 %[x], %[" S0 "], %[" S2 "], %[m] bitop3:0x78\n\t"                            \
  "v_bitop3_b32 %[F], %[x], %[" S1 "], %[" S2 "] bitop3:0xca\n\t"                            \
  "v_bitop3_b32 %[S], %[r1], %[r2], %[r3] bitop3:0x96\n\t"                                   \
  "v_add3_u32 %[G], %[S], %[F], %[" VI "]\n\t"                                               \
  "s_nop 1\n\t"                                                                              \
  "v_add_u32_dpp %[" NW "], %[G], %[G] row_shl:12 row_mask:0xf bank_mask:0xf bound_ctrl:1\n\t"

// Per-lane constants of the split round: rotation amounts and the side mask.
struct SplitLane {
  uint32_t c1, c2, c3, m;
};
// Working state of the split round (s3 only feeds the final sum).
struct SplitState {
  uint32_t s0, s1, s2, s3, v;
};

// Four rounds; k0..k3 are K + W of the round after each (1 on a-lanes).
__device__ __forceinline__ void split_rounds4(SplitState &q, uint32_t k0, uint32_t k1,
                                              uint32_t k2, uint32_t k3, const SplitLane &c) {
  uint32_t r1, r2, r3, x, F, S, G, P, v0, v1, v2, vo, n0, n1, n2, n3;
  asm volatile(EA_RND("s0", "s1", "s2", "k0", "V", "v0", "n0")
               EA_RND("n0", "s0", "s1", "k1", "v0", "v1", "n1")
               EA_RND("n1", "n0", "s0", "k2", "v1", "v2", "n2")
               EA_RND("n2", "n1", "n0", "k3", "v2", "Vo", "n3")
               : [r1] "=&v"(r1), [r2] "=&v"(r2), [r3] "=&v"(r3), [x] "=&v"(x), [F] "=&v"(F),
                 [S] "=&v"(S), [G] "=&v"(G), [P] "=&v"(P), [v0] "=&v"(v0), [v1] "=&v"(v1),
                 [v2] "=&v"(v2), [Vo] "=&v"(vo), [n0] "=&v"(n0), [n1] "=&v"(n1),
                 [n2] "=&v"(n2), [n3] "=&v"(n3)
               : [s0] "v"(q.s0), [s1] "v"(q.s1), [s2] "v"(q.s2), [V] "v"(q.v), [k0] "v"(k0),
                 [k1] "v"(k1), [k2] "v"(k2), [k3] "v"(k3), [c1] "v"(c.c1), [c2] "v"(c.c2),
                 [c3] "v"(c.c3), [m] "v"(c.m));
  q.s0 = n3; q.s1 = n2; q.s2 = n1; q.s3 = n0; q.v = vo;
}
// Three rounds.
__device__ __forceinline__ void split_rounds3(SplitState &q, uint32_t k0, uint32_t k1,
                                              uint32_t k2, const SplitLane &c) {
  uint32_t r1, r2, r3, x, F, S, G, P, v0, v1, vo, n0, n1, n2;
  asm volatile(EA_RND("s0", "s1", "s2", "k0", "V", "v0", "n0")
               EA_RND("n0", "s0", "s1", "k1", "v0", "v1", "n1")
               EA_RND("n1", "n0", "s0", "k2", "v1", "Vo", "n2")
               : [r1] "=&v"(r1), [r2] "=&v"(r2), [r3] "=&v"(r3), [x] "=&v"(x), [F] "=&v"(F),
                 [S] "=&v"(S), [G] "=&v"(G), [P] "=&v"(P), [v0] "=&v"(v0), [v1] "=&v"(v1),
                 [Vo] "=&v"(vo), [n0] "=&v"(n0), [n1] "=&v"(n1), [n2] "=&v"(n2)
               : [s0] "v"(q.s0), [s1] "v"(q.s1), [s2] "v"(q.s2), [V] "v"(q.v), [k0] "v"(k0),
                 [k1] "v"(k1), [k2] "v"(k2), [c1] "v"(c.c1), [c2] "v"(c.c2), [c3] "v"(c.c3),
                 [m] "v"(c.m));
  q.s3 = q.s0; q.s0 = n2; q.s1 = n1; q.s2 = n0; q.v = vo;
}
// Rounds 62 and 63 (the last): k0 is K + W of round 63.
__device__ __forceinline__ void split_rounds_end(SplitState &q, uint32_t k0,
                                                 const SplitLane &c) {
  uint32_t r1, r2, r3, x, F, S, G, P, v0, n0, n1;
  asm volatile(EA_RND("s0", "s1", "s2", "k0", "V", "v0", "n0")
               EA_RND_LAST("n0", "s0", "s1", "v0", "n1")
               : [r1] "=&v"(r1), [r2] "=&v"(r2), [r3] "=&v"(r3), [x] "=&v"(x), [F] "=&v"(F),
                 [S] "=&v"(S), [G] "=&v"(G), [P] "=&v"(P), [v0] "=&v"(v0), [n0] "=&v"(n0),
                 [n1] "=&v"(n1)
               : [s0] "v"(q.s0), [s1] "v"(q.s1), [s2] "v"(q.s2), [V] "v"(q.v), [k0] "v"(k0),
                 [c1] "v"(c.c1), [c2] "v"(c.c2), [c3] "v"(c.c3), [m] "v"(c.m));
  q.s3 = q.s1; q.s2 = q.s0; q.s1 = n0; q.s0 = n1;
}

// DPP move within a row of 16 lanes; lanes whose source lies outside the
// row read zero.
constexpr int kRowShl1 = 0x101, kRowShl9 = 0x109, kRowShl14 = 0x10E;
constexpr int kRowShr2 = 0x112, kRowShr7 = 0x117, kRowShr12 = 0x11C, kRowShr15 = 0x11F;
template <int CTRL>
__device__ __forceinline__ uint32_t row_move(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
__device__ __forceinline__ uint32_t sig0(uint32_t x) {
  return bitop3<kXor3>(rotr(x, 7), rotr(x, 18), x >> 3);
}
__device__ __forceinline__ uint32_t sig1(uint32_t x) {
  return bitop3<kXor3>(rotr(x, 17), rotr(x, 19), x >> 10);
}

// Lane j of a row holds W_T0-16+j; returns W_T0+j.
__device__ __forceinline__ uint32_t split_schedule16(uint32_t wp) {
  uint32_t q = sig0(row_move<kRowShl1>(wp)) + wp;  // sigma0(W_t-15) + W_t-16 (lane 15: below)
  q += row_move<kRowShl9>(wp);                      // W_t-7 for j < 7
  q += sig1(row_move<kRowShl14>(wp));               // sigma1(W_t-2) for j < 2
  uint32_t w = q;                                   // lanes 0, 1 final
  q += sig0(row_move<kRowShr15>(w));                // lane 15: sigma0(W_T0)
  uint32_t w1 = w, w2 = w;
#pragma unroll
  for (int s = 1; s < 8; ++s) {
    // lane j - 7 is final three steps before lane j
    const uint32_t t7 = row_move<kRowShr7>(w2) + q;
    w2 = w1; w1 = w;
    w = sig1(row_move<kRowShr2>(w)) + t7;
  }
  return w;
}

// LDS of the two-wave chain form, in 32-bit words.  Row r of both waves
// (16 lanes) carries the chain of sequence 4 * block + r: its K_t + W_t
// (t = 16..63) at kSpKw + 48 r, its last key and the 8 padding words of the
// chained block at kSpKey + 16 r; the 48 ones (the a-lanes' K + W) are
// shared; then a 4-word store slot for each lane that holds nothing
// (lanes 4..11 of each row).
constexpr int kSpRows = 4;
constexpr int kSpKw = 0;
constexpr int kSpOnes = kSpKw + 48 * kSpRows;
constexpr int kSpKey = kSpOnes + 48;
constexpr int kSpJunk = kSpKey + 16 * kSpRows;
constexpr int kSpWords = kSpJunk + 4 * 8 * kSpRows;

template <typename Off>
__global__ __launch_bounds__(128) void sha256_chain_split(
    const uint32_t *__restrict__ mid, const Off *__restrict__ key_off, int32_t n_seqs,
    uint32_t len_bits, const uint8_t *__restrict__ parents, uint8_t *__restrict__ keys) {
  __shared__ __align__(16) uint32_t lds[kSpWords];
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int j = lane & 15;
  const int row = lane >> 4;
  const bool e_lane = j >= 12;
  const bool a_lane = j < 4;
  // this row's sequence; rows past the last sequence carry an empty chain
  const int32_t s = (int32_t)blockIdx.x * kSpRows + row;
  int64_t k0 = 0, k1 = 0;
  if (s < n_seqs) {
    k0 = key_off[s];
    k1 = key_off[s + 1];
  }
  // Key counts in the offsets' width: with 32-bit offsets the loop and its
  // bounds stay 32-bit (scalar compares, one-instruction clamps).
  const Off len = (Off)(k1 - k0);
  // Every row of both waves runs the longest row's number of keys, so the
  // two waves meet at the same barriers; a row past its own end computes
  // keys that are never stored.
  Off kmax = 0;
#pragma unroll
  for (int r = 0; r < kSpRows; ++r) {
    Off l;
    if constexpr (sizeof(Off) == 4) {
      l = (Off)__builtin_amdgcn_readlane((int)len, 16 * r);
    } else {
      const uint32_t lo = __builtin_amdgcn_readlane((int)(uint32_t)len, 16 * r);
      const uint32_t hi = __builtin_amdgcn_readlane((int)(uint32_t)((uint64_t)len >> 32), 16 * r);
      l = (Off)(((uint64_t)hi << 32) | lo);
    }
    kmax = l > kmax ? l : kmax;
  }
  if (wave == 1) {
    if (lane < 48) lds[kSpOnes + lane] = 1u;
    if (j >= 8) lds[kSpKey + 16 * row + j] = j == 8 ? 0x80000000u : (j == 15 ? len_bits : 0u);
  }
  __syncthreads();
  if (wave == 0) {
    uint32_t prev[8];
    parent_words(s < n_seqs ? parents : nullptr, s, prev);
    SplitLane c;
    c.c1 = e_lane ? 6 : 2;
    c.c2 = e_lane ? 11 : 13;
    c.c3 = e_lane ? 25 : 22;
    c.m = e_lane ? 0u : 0xffffffffu;
    // K_t (t < 8) and K_t + W_t (t = 8..15, the padding) on e-lanes, 1 on a-lanes
    uint32_t kc[8], kwc[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) kc[t] = e_lane ? kRound[t] : 1u;
#pragma unroll
    for (int t = 8; t < 16; ++t) {
      const uint32_t w = t == 8 ? 0x80000000u : (t == 15 ? len_bits : 0u);
      kwc[t - 8] = e_lane ? kRound[t] + w : 1u;
    }
    uint32_t o[4];  // the previous key, this lane's half (a: H0..3, e: H4..7)
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = e_lane ? prev[4 + i] : prev[i];
    const int half = j >= 8 ? 1 : 0;
    // midstate of this row's key k0 + kk, held at the row's last key past
    // its end (key 0 for an empty row: some key exists whenever this runs)
    const uint4 *mbase = reinterpret_cast<const uint4 *>(mid) + 2 * (len > 0 ? k0 : 0) + half;
    const Off last = len > 0 ? len - 1 : 0;
    auto mid_at = [&](Off kk) { return mbase[2 * (int64_t)(kk < last ? kk : last)]; };
    uint4 nx = make_uint4(0, 0, 0, 0);
    if (kmax > 0) nx = mid_at(0);
    // The word offsets of the K + W reads and of the key store differ per
    // lane; hiding them keeps the compiler from reading both arrays and
    // selecting.
    uint32_t kbase = e_lane ? (uint32_t)(kSpKw + 48 * row) : (uint32_t)kSpOnes;
    asm volatile("" : "+v"(kbase));
    const uint4 *kw4 = reinterpret_cast<const uint4 *>(lds + kbase);
    uint32_t kst = a_lane ? (uint32_t)(kSpKey + 16 * row)
                          : (e_lane ? (uint32_t)(kSpKey + 16 * row + 4)
                                    : (uint32_t)(kSpJunk + 4 * (8 * row + j - 4)));
    asm volatile("" : "+v"(kst));
    uint4 *key_dst = reinterpret_cast<uint4 *>(lds + kst);
    for (Off kk = 0; kk < kmax; ++kk) {
      const uint4 h0 = nx;
      if (kk + 1 < kmax) nx = mid_at(kk + 1);
      SplitState q{h0.x, h0.y, h0.z, h0.w, 0u};
      uint32_t kw[8];  // K + W of rounds 0..7: the previous key
#pragma unroll
      for (int t = 0; t < 4; ++t) kw[t] = row_move<kRowShr12>(o[t]) + kc[t];
#pragma unroll
      for (int t = 4; t < 8; ++t) kw[t] = e_lane ? o[t - 4] + kc[t] : 1u;
      q.v = (q.s3 ^ c.m) + (row_move<kRowShr12>(q.s3) + kw[0]);
      split_rounds4(q, kw[1], kw[2], kw[3], kw[4], c);      // rounds 0..3
      split_rounds4(q, kw[5], kw[6], kw[7], kwc[0], c);     // 4..7
      split_rounds4(q, kwc[1], kwc[2], kwc[3], kwc[4], c);  // 8..11
      __syncthreads();
      uint4 a0 = kw4[0], a1 = kw4[1], a2 = kw4[2], a3 = kw4[3];  // t = 16..31
      split_rounds3(q, kwc[5], kwc[6], kwc[7], c);          // 12..14
      split_rounds4(q, a0.x, a0.y, a0.z, a0.w, c);          // 15..18
      split_rounds4(q, a1.x, a1.y, a1.z, a1.w, c);          // 19..22
      split_rounds4(q, a2.x, a2.y, a2.z, a2.w, c);          // 23..26
      __syncthreads();
      a0 = kw4[4]; a1 = kw4[5]; a2 = kw4[6];                // t = 32..43
      const uint4 b3 = kw4[7];                               // t = 44..47
      split_rounds4(q, a3.x, a3.y, a3.z, a3.w, c);          // 27..30
      split_rounds4(q, a0.x, a0.y, a0.z, a0.w, c);          // 31..34
      split_rounds4(q, a1.x, a1.y, a1.z, a1.w, c);          // 35..38
      split_rounds4(q, a2.x, a2.y, a2.z, a2.w, c);          // 39..42
      __syncthreads();
      a0 = kw4[8]; a1 = kw4[9]; a2 = kw4[10]; a3 = kw4[11];  // t = 48..63
      split_rounds4(q, b3.x, b3.y, b3.z, b3.w, c);          // 43..46
      split_rounds4(q, a0.x, a0.y, a0.z, a0.w, c);          // 47..50
      split_rounds4(q, a1.x, a1.y, a1.z, a1.w, c);          // 51..54
      split_rounds4(q, a2.x, a2.y, a2.z, a2.w, c);          // 55..58
      split_rounds3(q, a3.x, a3.y, a3.z, c);                // 59..61
      split_rounds_end(q, a3.w, c);                         // 62, 63
      o[0] = h0.x + q.s0; o[1] = h0.y + q.s1; o[2] = h0.z + q.s2; o[3] = h0.w + q.s3;
      *key_dst = make_uint4(o[0], o[1], o[2], o[3]);
      __syncthreads();
    }
  } else {
    // lane j: W_j of the first key's final block (the parent and padding),
    // read per lane rather than from prev[j], which a per-lane index would
    // move out of registers
    uint32_t wp = j == 8 ? 0x80000000u : (j == 15 ? len_bits : 0u);
    if (j < 8 && parents != nullptr && s < n_seqs) {
      const uint8_t *pw = parents + 32 * (int64_t)s + 4 * j;
      wp = ((uint32_t)pw[0] << 24) | ((uint32_t)pw[1] << 16) | ((uint32_t)pw[2] << 8) | pw[3];
    }
    const uint32_t kp0 = kRound[16 + j], kp1 = kRound[32 + j], kp2 = kRound[48 + j];
    uint32_t *kw_row = lds + kSpKw + 48 * row;
    for (Off kk = 0; kk < kmax; ++kk) {
      const uint32_t key_prev = wp;  // lanes 0..7: key kk - 1 of this row
      uint32_t w = split_schedule16(wp);
      kw_row[j] = w + kp0;
      __syncthreads();
      if (kk > 0 && kk <= len && j < 8)
        reinterpret_cast<uint32_t *>(keys + 32 * (k0 + (int64_t)kk - 1))[j] = __builtin_bswap32(key_prev);
      w = split_schedule16(w);
      kw_row[16 + j] = w + kp1;
      __syncthreads();
      w = split_schedule16(w);
      kw_row[32 + j] = w + kp2;
      __syncthreads();
      __syncthreads();
      wp = lds[kSpKey + 16 * row + j];
    }
    // a row as long as the longest stores its last key here; shorter rows
    // stored theirs in the loop
    if (len > 0 && len == kmax && j < 8)
      reinterpret_cast<uint32_t *>(keys + 32 * (k1 - 1))[j] = __builtin_bswap32(wp);
  }
}

// Midstates of few keys with several token blocks each: a workgroup of two
// waves per four keys, row r (16 lanes) of both waves on key 4 * block + r.
// The token blocks of a key are compressed one after the other, but their
// message schedules depend on the tokens alone, so wave 1 prepares block
// c + 1's 64 words (K_t + W_t) for every row in one half of an LDS double
// buffer while wave 0 runs block c's 64 rounds in the split form of the
// chain kernel above from the other half: one barrier per block, and every
// key of a launch has the same number of blocks, so the rows stay in step.
// Rows past the last key rerun row 0's tokens and store nothing.
//
// LDS in 32-bit words: two halves of kMsHalf words, row r's K_t + W_t at
// 64 r of each, then the 64 ones the a-lanes read as their K + W.
constexpr int kMsHalf = 64 * kSpRows;
constexpr int kMsOnes = 2 * kMsHalf;
constexpr int kMsWords = kMsOnes + 64;

template <typename Off>
__global__ __launch_bounds__(128) void sha256_midstates_split(
    const int32_t *__restrict__ tokens, const Off *__restrict__ key_off,
    const Off *__restrict__ tok_off, int32_t n_seqs, int64_t n_keys, int32_t block_tokens,
    uint32_t *__restrict__ mid) {
  __shared__ __align__(16) uint32_t lds[kMsWords];
  const int wave = __builtin_amdgcn_readfirstlane((int)threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int j = lane & 15;
  const int row = lane >> 4;
  const bool e_lane = j >= 12;
  const int64_t lim = n_keys < (int64_t)key_off[n_seqs] ? n_keys : (int64_t)key_off[n_seqs];
  const int64_t g0 = (int64_t)blockIdx.x * kSpRows;
  if (g0 >= lim) return;  // the whole workgroup
  const int32_t s0 = owner(key_off, n_seqs, g0);
  if (g0 < (int64_t)key_off[s0] || g0 >= (int64_t)key_off[s0 + 1]) return;  // the whole workgroup
  const int32_t *tok =
      tokens + (int64_t)tok_off[s0] + (g0 - (int64_t)key_off[s0]) * block_tokens;
  const int64_t g = g0 + row;
  bool ok = false;
  if (row > 0 && g < lim) {
    const int32_t s = owner(key_off, n_seqs, g);
    if (g >= (int64_t)key_off[s] && g < (int64_t)key_off[s + 1]) {
      ok = true;
      tok = tokens + (int64_t)tok_off[s] + (g - (int64_t)key_off[s]) * block_tokens;
    }
  }
  ok = ok || row == 0;
  const int32_t blocks = block_tokens / 16;
  if (wave == 1) {
    // lane j of row r: word j of the row's current block, W_16+j, W_32+j and
    // W_48+j in turn; the next block's token read one block ahead
    lds[kMsOnes + lane] = 1u;
    const uint32_t kp0 = kRound[j], kp1 = kRound[16 + j], kp2 = kRound[32 + j],
                   kp3 = kRound[48 + j];
    uint32_t nx = (uint32_t)tok[j];
    for (int32_t c = 0; c < blocks; ++c) {
      uint32_t w = __builtin_bswap32(nx);  // LE32 token bytes read as a big-endian word
      if (c + 1 < blocks) nx = (uint32_t)tok[16 * (c + 1) + j];
      uint32_t *kw_row = lds + (c & 1) * kMsHalf + 64 * row;
      kw_row[j] = w + kp0;
      w = split_schedule16(w);
      kw_row[16 + j] = w + kp1;
      w = split_schedule16(w);
      kw_row[32 + j] = w + kp2;
      w = split_schedule16(w);
      kw_row[48 + j] = w + kp3;
      __syncthreads();
    }
    __syncthreads();  // the rounds wave's last block
  } else {
    SplitLane c;
    c.c1 = e_lane ? 6 : 2;
    c.c2 = e_lane ? 11 : 13;
    c.c3 = e_lane ? 25 : 22;
    c.m = e_lane ? 0u : 0xffffffffu;
    uint32_t h0 = e_lane ? kInit[4] : kInit[0], h1 = e_lane ? kInit[5] : kInit[1];
    uint32_t h2 = e_lane ? kInit[6] : kInit[2], h3 = e_lane ? kInit[7] : kInit[3];
    // e-lanes read their row's words in the current half, the other lanes
    // the ones; hidden from the compiler, which would otherwise read both
    // and select
    uint32_t kbase = e_lane ? (uint32_t)(64 * row) : (uint32_t)kMsOnes;
    uint32_t kstep = e_lane ? (uint32_t)kMsHalf : 0u;
    asm volatile("" : "+v"(kbase), "+v"(kstep));
    __syncthreads();  // block 0's words
    for (int32_t cb = 0; cb < blocks; ++cb) {
      const uint4 *kw4 = reinterpret_cast<const uint4 *>(lds + kbase + (cb & 1) * kstep);
      uint32_t kw[64];
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const uint4 v = kw4[i];
        kw[4 * i] = v.x; kw[4 * i + 1] = v.y; kw[4 * i + 2] = v.z; kw[4 * i + 3] = v.w;
      }
      SplitState q{h0, h1, h2, h3, 0u};
      q.v = (q.s3 ^ c.m) + (row_move<kRowShr12>(q.s3) + kw[0]);
#pragma unroll
      for (int t = 0; t < 56; t += 4)  // rounds 0..55
        split_rounds4(q, kw[t + 1], kw[t + 2], kw[t + 3], kw[t + 4], c);
      split_rounds3(q, kw[57], kw[58], kw[59], c);  // 56..58
      split_rounds3(q, kw[60], kw[61], kw[62], c);  // 59..61
      split_rounds_end(q, kw[63], c);               // 62, 63
      h0 += q.s0; h1 += q.s1; h2 += q.s2; h3 += q.s3;
      __syncthreads();
    }
    if (ok && (j == 0 || j == 12))
      reinterpret_cast<uint4 *>(mid + 8 * g)[e_lane ? 1 : 0] = make_uint4(h0, h1, h2, h3);
  }
}

// One lane per sequence: the working state and the message schedule of a
// chained compression all in one lane.  Message words 8..15 are the fixed
// padding of a 32-byte parent (the 0x80 byte, zeros, the bit length).
template <typename Off>
__global__ __launch_bounds__(256) void sha256_chain_lane(
    const uint32_t *__restrict__ mid, const Off *__restrict__ key_off,
    int32_t n_seqs, uint32_t len_bits, const uint8_t *__restrict__ parents,
    uint8_t *__restrict__ keys) {
  const int32_t s = blockIdx.x * 256 + threadIdx.x;
  if (s >= n_seqs) return;
  uint32_t prev[8];
  parent_words(parents, s, prev);
  const int64_t k0 = key_off[s], k1 = key_off[s + 1];
  const uint4 *mh = reinterpret_cast<const uint4 *>(mid);
  uint4 n0 = make_uint4(0, 0, 0, 0), n1 = n0;
  if (k0 < k1) {
    n0 = mh[2 * k0];
    n1 = mh[2 * k0 + 1];
  }
  // first midstate taken before the loop, as in the two-lane form
  asm volatile("" ::"v"(n0.x), "v"(n0.y), "v"(n0.z), "v"(n0.w), "v"(n1.x), "v"(n1.y),
               "v"(n1.z), "v"(n1.w));
  for (int64_t k = k0; k < k1; ++k) {
    uint32_t st[8] = {n0.x, n0.y, n0.z, n0.w, n1.x, n1.y, n1.z, n1.w};
    if (k + 1 < k1) {
      n0 = mh[2 * (k + 1)];
      n1 = mh[2 * (k + 1) + 1];
    }
    uint32_t w[16];
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = prev[j];
    w[8] = 0x80000000u;
#pragma unroll
    for (int j = 9; j < 15; ++j) w[j] = 0u;
    w[15] = len_bits;
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

// Key offsets from device-resident sequence offsets, in two kernels.  A
// workgroup owns kScanSeqs consecutive sequences, kScanRun per thread
// (thread t the t-th run), so its loads cover one contiguous range.  Each
// group also records where each of its sub-blocks of kSubSeqs sequences
// starts inside it, for the fused hash kernel, whose workgroups are those
// sub-blocks (one sequence per lane).
//   hash_offsets_partials: each workgroup counts the full blocks of its
//     sequences and checks them; the last workgroup to finish (a ticket
//     counter, reset by that workgroup) turns the per-workgroup totals into
//     exclusive prefixes, the grand total and an error flag.
//   hash_offsets_write: each workgroup scans its own counts from its prefix
//     and writes key_off_out (int64, the caller's) and the kernels' copies
//     koff / toff in Off.
// Invalid offsets (a negative start, a decrease, an end past n_tokens) or
// more keys than keys_cap: key_off_out[0] = -1 and koff all zero, so the
// hash kernels that follow write nothing.
constexpr int kScanThreads = 256;
constexpr int kScanRun = 8;
constexpr int64_t kScanSeqs = (int64_t)kScanThreads * kScanRun;
constexpr int kSubSeqs = 256;
constexpr int kSubThreads = kSubSeqs / kScanRun;  // scan threads per sub-block
constexpr int kSubsPerGroup = (int)(kScanSeqs / kSubSeqs);
static_assert(kScanSeqs == kHashScanSeqs && kSubSeqs == kHashScanSub,
              "scan groups and the scratch's scan state agree");

// Scan state in device memory: [0] ticket counter (zero between calls),
// [1] grand total, [2] error flag, then per workgroup its total and, after
// the last workgroup's pass, its exclusive prefix, then per sub-block its
// exclusive prefix inside its group.
struct ScanState {
  uint64_t *ticket;
  int64_t *total;
  int64_t *bad;
  int64_t *part;    // [groups]
  int64_t *prefix;  // [groups]
  int64_t *subex;   // [groups * kSubsPerGroup]
};

__device__ __forceinline__ int64_t full_blocks(int64_t len, int32_t block_tokens, int32_t shift) {
  return shift >= 0 ? (len >> shift) : len / block_tokens;
}

// This thread's run: sequences [s0, s1), their offsets loaded together.
struct Run {
  int64_t s0, s1;
  int64_t off[kScanRun + 1];
};

__device__ __forceinline__ void load_run(const int64_t *seq_off, int32_t n_seqs, Run &r) {
  r.s0 = min((int64_t)blockIdx.x * kScanSeqs + (int64_t)threadIdx.x * kScanRun, (int64_t)n_seqs);
  r.s1 = min(r.s0 + kScanRun, (int64_t)n_seqs);
#pragma unroll
  for (int j = 0; j <= kScanRun; ++j) r.off[j] = r.s0 + j <= r.s1 ? seq_off[r.s0 + j] : 0;
}

constexpr int kScanWaves = kScanThreads / 64;

// Inclusive scan of v over the workgroup: within each wave by lane shifts
// (no barrier), then across the waves through their totals in lds (one
// barrier).  *total gets the workgroup's sum.  lds holds kScanWaves
// entries; the call ends with a barrier, so it can be reused at once.
__device__ __forceinline__ int64_t group_scan(int64_t v, int64_t *lds, int64_t *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int d = 1; d < 64; d <<= 1) {
    const int64_t t = __shfl_up(v, (unsigned)d, 64);
    if (lane >= d) v += t;
  }
  if (lane == 63) lds[wave] = v;
  __syncthreads();
  int64_t before = 0, all = 0;
#pragma unroll
  for (int w = 0; w < kScanWaves; ++w) {
    const int64_t t = lds[w];
    before += w < wave ? t : 0;
    all += t;
  }
  __syncthreads();
  *total = all;
  return v + before;
}

// Sum over the workgroup of v (every thread returns it).
__device__ __forceinline__ int64_t group_sum(int64_t v, int64_t *lds) {
  int64_t total;
  (void)group_scan(v, lds, &total);
  return total;
}

__global__ __launch_bounds__(kScanThreads) void hash_offsets_partials(
    const int64_t *__restrict__ seq_off, int32_t n_seqs, int64_t n_tokens, int32_t block_tokens,
    int32_t shift, ScanState st) {
  __shared__ int64_t lds[kScanWaves];
  __shared__ bool last;
  Run r;
  load_run(seq_off, n_seqs, r);
  bool ok = !(blockIdx.x == 0 && threadIdx.x == 0) || (r.off[0] >= 0 && r.off[0] <= n_tokens);
  int64_t count = 0;
#pragma unroll
  for (int j = 0; j < kScanRun; ++j)
    if (r.s0 + j < r.s1) {
      const int64_t a = r.off[j], e = r.off[j + 1];
      ok = ok && e >= a && e <= n_tokens;
      count += ok ? full_blocks(e - a, block_tokens, shift) : 0;
    }
  int64_t sum;
  const int64_t before = group_scan(count, lds, &sum) - count;
  if (threadIdx.x % kSubThreads == 0)  // where this thread's sub-block starts
    st.subex[(int64_t)blockIdx.x * kSubsPerGroup + threadIdx.x / kSubThreads] = before;
  const int64_t nbad = group_sum(ok ? 0 : 1, lds);
  if (threadIdx.x == 0) {
    st.part[blockIdx.x] = nbad ? -1 : sum;
    // publish this workgroup's total, then take a ticket; the last ticket
    // sees every total (release / acquire at device scope)
    const uint64_t t = __hip_atomic_fetch_add(st.ticket, 1ull, __ATOMIC_ACQ_REL,
                                              __HIP_MEMORY_SCOPE_AGENT);
    last = t == gridDim.x - 1;
  }
  __syncthreads();
  if (!last) return;
  // the last workgroup: exclusive prefixes of the totals, in order
  const int64_t groups = gridDim.x;
  const int64_t per = (groups + kScanThreads - 1) / kScanThreads;
  const int64_t g0 = min((int64_t)threadIdx.x * per, groups), g1 = min(g0 + per, groups);
  int64_t mine = 0, bad = 0;
  for (int64_t g = g0; g < g1; ++g) {
    const int64_t v = __hip_atomic_load(st.part + g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    bad |= v < 0;
    mine += v < 0 ? 0 : v;
  }
  int64_t total;
  int64_t run = group_scan(mine, lds, &total) - mine;  // exclusive prefix of the thread sums
  for (int64_t g = g0; g < g1; ++g) {
    st.prefix[g] = run;
    const int64_t v = __hip_atomic_load(st.part + g, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    run += v < 0 ? 0 : v;
  }
  const int64_t any_bad = group_sum(bad, lds);
  if (threadIdx.x == kScanThreads - 1) {
    *st.total = total;
    *st.bad = any_bad;
    // ready for the next call (stream order keeps calls apart)
    __hip_atomic_store(st.ticket, 0ull, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <typename Off>
__global__ __launch_bounds__(kScanThreads) void hash_offsets_write(
    const int64_t *__restrict__ seq_off, int32_t n_seqs, int32_t block_tokens, int32_t shift,
    int64_t keys_cap, ScanState st, int64_t *__restrict__ key_off_out, Off *__restrict__ koff,
    Off *__restrict__ toff) {
  __shared__ int64_t lds[kScanWaves];
  Run r;
  load_run(seq_off, n_seqs, r);
  const int64_t total = *st.total;
  const bool failed = *st.bad != 0 || total > keys_cap;
  const bool tail = blockIdx.x == gridDim.x - 1 && threadIdx.x == kScanThreads - 1;
  if (failed) {
    if (blockIdx.x == 0 && threadIdx.x == 0) key_off_out[0] = -1;
    for (int64_t s = r.s0; s < r.s1; ++s) koff[s] = 0;
    if (tail) koff[n_seqs] = 0;
    return;
  }
  int64_t cnt[kScanRun];
  int64_t mine = 0;
#pragma unroll
  for (int j = 0; j < kScanRun; ++j) {
    cnt[j] = r.s0 + j < r.s1 ? full_blocks(r.off[j + 1] - r.off[j], block_tokens, shift) : 0;
    mine += cnt[j];
  }
  int64_t group_total;
  int64_t run = st.prefix[blockIdx.x] + group_scan(mine, lds, &group_total) - mine;
#pragma unroll
  for (int j = 0; j < kScanRun; ++j)
    if (r.s0 + j < r.s1) {
      key_off_out[r.s0 + j] = run;
      koff[r.s0 + j] = (Off)run;
      toff[r.s0 + j] = (Off)r.off[j];
      run += cnt[j];
    }
  if (tail) {
    key_off_out[n_seqs] = total;
    koff[n_seqs] = (Off)total;
  }
}

// Zero the scan's ticket counter (a fill kernel rather than a memset, so
// that a captured graph replays it safely).
__global__ __launch_bounds__(64) void hash_scan_reset(uint64_t *ticket) {
  if (threadIdx.x == 0) *ticket = 0;
}

// One lane per sequence for the whole key: the token blocks of a key from
// the initial hash value, then the chained block, key after key, with the
// next token block loaded while the current one is compressed.  For batches
// of at least one wave of sequences per SIMD this leaves out the midstates'
// trip through memory and the second launch.
template <typename Off>
__global__ __launch_bounds__(256) void sha256_fused_lane(
    const int32_t *__restrict__ tokens, const Off *__restrict__ key_off,
    const Off *__restrict__ tok_off, int32_t n_seqs, int32_t block_tokens, uint32_t len_bits,
    const uint8_t *__restrict__ parents, uint8_t *__restrict__ keys) {
  const int32_t s = blockIdx.x * 256 + threadIdx.x;
  if (s >= n_seqs) return;
  uint32_t prev[8];
  parent_words(parents, s, prev);
  const int64_t k0 = key_off[s], k1 = key_off[s + 1];
  const int32_t blocks = block_tokens / 16;
  const int64_t total = (k1 - k0) * blocks;  // token blocks of the sequence
  const int32_t *tok = tokens + (int64_t)tok_off[s];
  uint32_t nx[16];
  if (total > 0)
#pragma unroll
    for (int j = 0; j < 16; ++j) nx[j] = (uint32_t)tok[j];
  int64_t q = 0;  // token blocks consumed
  for (int64_t k = k0; k < k1; ++k) {
    uint32_t st[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) st[j] = kInit[j];
    for (int32_t c = 0; c < blocks; ++c, ++q) {
      uint32_t w[16];
#pragma unroll
      for (int j = 0; j < 16; ++j)  // LE32 token bytes read as a big-endian word
        w[j] = __builtin_bswap32(nx[j]);
      if (q + 1 < total)
#pragma unroll
        for (int j = 0; j < 16; ++j) nx[j] = (uint32_t)tok[16 * (q + 1) + j];
      compress(st, w);
    }
    uint32_t w[16];
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = prev[j];
    w[8] = 0x80000000u;
#pragma unroll
    for (int j = 9; j < 15; ++j) w[j] = 0u;
    w[15] = len_bits;
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

// The fused form with the key offsets derived in the same kernel: workgroup
// b holds the scan's sub-block b (one sequence per lane), so it turns its
// counts of full blocks into key offsets from the prefixes the scan's first
// kernel left for the group and the sub-block, writes them for the caller
// and hashes.  The first token block is requested before the scan, so the
// scan runs while it arrives.  On a failed scan (invalid offsets, too many
// keys) it writes key_off_out[0] = -1 and nothing else.
__global__ __launch_bounds__(kSubSeqs) void sha256_fused_scan(
    const int32_t *__restrict__ tokens, const int64_t *__restrict__ seq_off, int32_t n_seqs,
    int32_t block_tokens, int32_t shift, int64_t keys_cap, uint32_t len_bits, ScanState st,
    int64_t *__restrict__ key_off_out, const uint8_t *__restrict__ parents,
    uint8_t *__restrict__ keys) {
  __shared__ int64_t lds[kScanWaves];
  const int64_t total = *st.total;
  if (*st.bad != 0 || total > keys_cap) {  // the same for every work-item
    if (blockIdx.x == 0 && threadIdx.x == 0) key_off_out[0] = -1;
    return;
  }
  const int32_t s = blockIdx.x * kSubSeqs + threadIdx.x;
  const bool live = s < n_seqs;
  const int64_t a = live ? seq_off[s] : 0;
  const int64_t cnt = live ? full_blocks(seq_off[s + 1] - a, block_tokens, shift) : 0;
  const int32_t *tok = tokens + a;
  uint32_t nx[16];
  if (cnt > 0)
#pragma unroll
    for (int j = 0; j < 16; ++j) nx[j] = (uint32_t)tok[j];
  int64_t sub_total;
  const int64_t k0 = st.prefix[blockIdx.x / kSubsPerGroup] + st.subex[blockIdx.x] +
                     group_scan(cnt, lds, &sub_total) - cnt;
  if (!live) return;
  key_off_out[s] = k0;
  if (s == n_seqs - 1) key_off_out[n_seqs] = total;
  if (cnt == 0) return;
  uint32_t prev[8];
  parent_words(parents, s, prev);
  const int32_t blocks = block_tokens / 16;
  const int64_t nblk = cnt * blocks;  // token blocks of the sequence
  int64_t q = 0;  // token blocks consumed
  for (int64_t k = k0; k < k0 + cnt; ++k) {
    uint32_t st8[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) st8[j] = kInit[j];
    for (int32_t c = 0; c < blocks; ++c, ++q) {
      uint32_t w[16];
#pragma unroll
      for (int j = 0; j < 16; ++j)  // LE32 token bytes read as a big-endian word
        w[j] = __builtin_bswap32(nx[j]);
      if (q + 1 < nblk)
#pragma unroll
        for (int j = 0; j < 16; ++j) nx[j] = (uint32_t)tok[16 * (q + 1) + j];
      compress(st8, w);
    }
    uint32_t w[16];
#pragma unroll
    for (int j = 0; j < 8; ++j) w[j] = prev[j];
    w[8] = 0x80000000u;
#pragma unroll
    for (int j = 9; j < 15; ++j) w[j] = 0u;
    w[15] = len_bits;
    compress(st8, w);
    uint4 *out = reinterpret_cast<uint4 *>(keys + 32 * k);
    out[0] = make_uint4(__builtin_bswap32(st8[0]), __builtin_bswap32(st8[1]),
                        __builtin_bswap32(st8[2]), __builtin_bswap32(st8[3]));
    out[1] = make_uint4(__builtin_bswap32(st8[4]), __builtin_bswap32(st8[5]),
                        __builtin_bswap32(st8[6]), __builtin_bswap32(st8[7]));
#pragma unroll
    for (int j = 0; j < 8; ++j) prev[j] = st8[j];
  }
}

// The split forms launch one workgroup per four keys (midstates) or four
// sequences (chain); forcing them on more than this many workgroups falls
// back to the other forms.
constexpr int64_t kMaxSplitGroups = int64_t(1) << 24;

// Compute units of the current device, cached per device.
hipError_t device_cus(int *out) {
  static std::atomic<int> cache[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev >= 0 && dev < 64 && cache[dev].load(std::memory_order_relaxed) > 0) {
    *out = cache[dev].load(std::memory_order_relaxed);
    return hipSuccess;
  }
  int cus = 0;
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return e;
  *out = cus > 0 ? cus : 1;
  if (dev >= 0 && dev < 64) cache[dev].store(*out, std::memory_order_relaxed);
  return hipSuccess;
}

}  // namespace

hipError_t launch_sha256_midstates(const int32_t *d_tokens, const void *d_key_offsets,
                                   const void *d_tok_offsets, bool wide, int32_t n_seqs,
                                   int64_t n_keys, int32_t block_tokens, uint32_t *d_mid,
                                   hipStream_t stream) {
  if (n_keys <= 0) return hipSuccess;
  // Keys of several blocks, at most 16 per compute unit (8 for two-block
  // keys, where the lane form catches up sooner): a workgroup of two waves
  // per four keys (the schedules on their own wave); otherwise one lane per
  // key.  EA_HASH_MID=lane or split forces a form.
  const int64_t groups = (n_keys + kSpRows - 1) / kSpRows;
  bool split = false;
  const char *f = std::getenv("EA_HASH_MID");
  if (f && std::strcmp(f, "split") == 0) {
    split = groups <= kMaxSplitGroups;
  } else if (!(f && std::strcmp(f, "lane") == 0) && block_tokens >= 32) {
    int cus = 0;
    const hipError_t e = device_cus(&cus);
    if (e != hipSuccess) return e;
    split = n_keys <= (block_tokens >= 64 ? 16 : 8) * (int64_t)cus;
  }
  (void)hipGetLastError();  // report this launch's status only
  const int64_t blocks = (n_keys + 255) / 256;
  if (split && wide)
    hipLaunchKernelGGL(sha256_midstates_split<int64_t>, dim3((unsigned)groups), dim3(128), 0,
                       stream, d_tokens, static_cast<const int64_t *>(d_key_offsets),
                       static_cast<const int64_t *>(d_tok_offsets), n_seqs, n_keys,
                       block_tokens, d_mid);
  else if (split)
    hipLaunchKernelGGL(sha256_midstates_split<int32_t>, dim3((unsigned)groups), dim3(128), 0,
                       stream, d_tokens, static_cast<const int32_t *>(d_key_offsets),
                       static_cast<const int32_t *>(d_tok_offsets), n_seqs, n_keys,
                       block_tokens, d_mid);
  else if (wide)
    hipLaunchKernelGGL(sha256_midstates<int64_t>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       d_tokens, static_cast<const int64_t *>(d_key_offsets),
                       static_cast<const int64_t *>(d_tok_offsets), n_seqs, n_keys,
                       block_tokens, d_mid);
  else
    hipLaunchKernelGGL(sha256_midstates<int32_t>, dim3((unsigned)blocks), dim3(256), 0, stream,
                       d_tokens, static_cast<const int32_t *>(d_key_offsets),
                       static_cast<const int32_t *>(d_tok_offsets), n_seqs, n_keys,
                       block_tokens, d_mid);
  return hipGetLastError();
}

namespace {

enum ChainForm { kChainPair = 0, kChainLane = 1, kChainSplit = 2 };

template <typename Off>
void launch_chain(int form, const uint32_t *d_mid, const Off *d_koff, int32_t n_seqs,
                  uint32_t len_bits, const uint8_t *d_parents, uint8_t *d_keys,
                  hipStream_t stream) {
  if (form == kChainLane)
    hipLaunchKernelGGL(sha256_chain_lane<Off>, dim3((n_seqs + 255) / 256), dim3(256), 0, stream,
                       d_mid, d_koff, n_seqs, len_bits, d_parents, d_keys);
  else if (form == kChainSplit)
    hipLaunchKernelGGL(sha256_chain_split<Off>, dim3((n_seqs + kSpRows - 1) / kSpRows),
                       dim3(128), 0, stream, d_mid, d_koff, n_seqs, len_bits, d_parents, d_keys);
  else
    hipLaunchKernelGGL(sha256_chain<Off>, dim3((n_seqs + 31) / 32), dim3(64), 0, stream, d_mid,
                       d_koff, n_seqs, len_bits, d_parents, d_keys);
}

}  // namespace

hipError_t launch_sha256_chain(const uint32_t *d_mid, const void *d_key_offsets, bool wide,
                               int32_t n_seqs, int32_t block_tokens, const uint8_t *d_parents,
                               uint8_t *d_keys, hipStream_t stream) {
  if (n_seqs <= 0) return hipSuccess;
  // message = 4b token bytes + 32 key bytes
  const uint32_t len_bits = (uint32_t)(8u * (4u * (uint32_t)block_tokens + 32u));
  int form = -1;
  if (const char *f = std::getenv("EA_HASH_CHAIN")) {  // forces a form
    if (std::strcmp(f, "pair") == 0) form = kChainPair;
    if (std::strcmp(f, "lane") == 0) form = kChainLane;
    if (std::strcmp(f, "split") == 0) form = kChainSplit;
  }
  if (form == kChainSplit && n_seqs > kMaxSplitGroups) form = kChainPair;  // grid bound
  if (form < 0) {
    // Up to eight sequences per compute unit (two workgroups of four rows):
    // the split form, 4-30% less time per call than two lanes per sequence
    // for chains of 16 to 1,024 keys (1,024 chains of 1,024 keys: 1.55
    // against 2.15 ms).  At sixteen per compute unit the two-lane form wins
    // for long chains (its waves hold 32 chains each), beyond for all, and
    // beyond 128 per compute unit one lane per sequence does.
    int cus = 0;
    const hipError_t e = device_cus(&cus);
    if (e != hipSuccess) return e;
    form = (int64_t)n_seqs <= 8 * (int64_t)cus
               ? kChainSplit
               : ((int64_t)n_seqs > 128 * (int64_t)cus ? kChainLane : kChainPair);
  }
  (void)hipGetLastError();  // report this launch's status only
  if (wide)
    launch_chain(form, d_mid, static_cast<const int64_t *>(d_key_offsets), n_seqs, len_bits,
                 d_parents, d_keys, stream);
  else
    launch_chain(form, d_mid, static_cast<const int32_t *>(d_key_offsets), n_seqs, len_bits,
                 d_parents, d_keys, stream);
  return hipGetLastError();
}

bool hash_fused(int32_t n_seqs) {
  const char *f = std::getenv("EA_HASH_CHAIN");
  if (f && *f) return std::strcmp(f, "fused") == 0;
  int cus = 0;
  if (device_cus(&cus) != hipSuccess) return false;
  // at least one wave of sequences on every SIMD (four per compute unit)
  return (int64_t)n_seqs >= 256 * (int64_t)cus;
}

hipError_t launch_sha256_fused(const int32_t *d_tokens, const void *d_key_offsets,
                               const void *d_tok_offsets, bool wide, int32_t n_seqs,
                               int32_t block_tokens, const uint8_t *d_parents, uint8_t *d_keys,
                               hipStream_t stream) {
  if (n_seqs <= 0) return hipSuccess;
  const uint32_t len_bits = (uint32_t)(8u * (4u * (uint32_t)block_tokens + 32u));
  (void)hipGetLastError();
  const dim3 g((unsigned)((n_seqs + 255) / 256));
  if (wide)
    hipLaunchKernelGGL(sha256_fused_lane<int64_t>, g, dim3(256), 0, stream, d_tokens,
                       static_cast<const int64_t *>(d_key_offsets),
                       static_cast<const int64_t *>(d_tok_offsets), n_seqs, block_tokens,
                       len_bits, d_parents, d_keys);
  else
    hipLaunchKernelGGL(sha256_fused_lane<int32_t>, g, dim3(256), 0, stream, d_tokens,
                       static_cast<const int32_t *>(d_key_offsets),
                       static_cast<const int32_t *>(d_tok_offsets), n_seqs, block_tokens,
                       len_bits, d_parents, d_keys);
  return hipGetLastError();
}

hipError_t launch_hash_scan_reset(void *d_state, hipStream_t stream) {
  (void)hipGetLastError();
  hipLaunchKernelGGL(hash_scan_reset, dim3(1), dim3(64), 0, stream,
                     static_cast<uint64_t *>(d_state));
  return hipGetLastError();
}

int64_t hash_scan_groups(int32_t n_seqs) {
  return std::max<int64_t>(1, ((int64_t)n_seqs + kScanSeqs - 1) / kScanSeqs);
}

// The scan state's fields inside d_state (see ScanState).
ScanState scan_state(void *d_state, int64_t groups) {
  uint8_t *base = static_cast<uint8_t *>(d_state);
  int64_t *words = reinterpret_cast<int64_t *>(base + 64);
  return ScanState{reinterpret_cast<uint64_t *>(base), reinterpret_cast<int64_t *>(base + 8),
                   reinterpret_cast<int64_t *>(base + 16), words, words + groups,
                   words + 2 * groups};
}

int block_shift(int32_t block_tokens) {
  return (block_tokens & (block_tokens - 1)) == 0 ? __builtin_ctz(block_tokens) : -1;
}

hipError_t launch_hash_key_offsets(const int64_t *d_seq_offsets, int32_t n_seqs,
                                   int64_t n_tokens, int32_t block_tokens, int64_t keys_cap,
                                   int64_t *d_key_offsets_out, bool wide, void *d_koff,
                                   void *d_toff, void *d_state, hipStream_t stream) {
  const int shift = block_shift(block_tokens);
  const int64_t groups = hash_scan_groups(n_seqs);
  const ScanState st = scan_state(d_state, groups);
  (void)hipGetLastError();  // report this launch's status only
  hipLaunchKernelGGL(hash_offsets_partials, dim3((unsigned)groups), dim3(kScanThreads), 0, stream,
                     d_seq_offsets, n_seqs, n_tokens, block_tokens, shift, st);
  if (wide)
    hipLaunchKernelGGL(hash_offsets_write<int64_t>, dim3((unsigned)groups), dim3(kScanThreads), 0,
                       stream, d_seq_offsets, n_seqs, block_tokens, shift, keys_cap, st,
                       d_key_offsets_out, static_cast<int64_t *>(d_koff),
                       static_cast<int64_t *>(d_toff));
  else
    hipLaunchKernelGGL(hash_offsets_write<int32_t>, dim3((unsigned)groups), dim3(kScanThreads), 0,
                       stream, d_seq_offsets, n_seqs, block_tokens, shift, keys_cap, st,
                       d_key_offsets_out, static_cast<int32_t *>(d_koff),
                       static_cast<int32_t *>(d_toff));
  return hipGetLastError();
}

hipError_t launch_hash_fused_offsets(const int32_t *d_tokens, const int64_t *d_seq_offsets,
                                     int32_t n_seqs, int64_t n_tokens, int32_t block_tokens,
                                     int64_t keys_cap, int64_t *d_key_offsets_out,
                                     const uint8_t *d_parents, uint8_t *d_keys, void *d_state,
                                     hipStream_t stream) {
  const int shift = block_shift(block_tokens);
  const int64_t groups = hash_scan_groups(n_seqs);
  const ScanState st = scan_state(d_state, groups);
  const uint32_t len_bits = (uint32_t)(8u * (4u * (uint32_t)block_tokens + 32u));
  (void)hipGetLastError();
  hipLaunchKernelGGL(hash_offsets_partials, dim3((unsigned)groups), dim3(kScanThreads), 0, stream,
                     d_seq_offsets, n_seqs, n_tokens, block_tokens, shift, st);
  const int64_t subs = ((int64_t)n_seqs + kSubSeqs - 1) / kSubSeqs;
  hipLaunchKernelGGL(sha256_fused_scan, dim3((unsigned)subs), dim3(kSubSeqs), 0, stream,
                     d_tokens, d_seq_offsets, n_seqs, block_tokens, shift, keys_cap, len_bits, st,
                     d_key_offsets_out, d_parents, d_keys);
  return hipGetLastError();
}

// Fixed device memory for the hashing entry point that allocates nothing
// (layout in ea_internal.hpp).  Each device holds its own copy for the
// life of the process.  In host code the array's name is not a device
// address: the address comes from hipGetSymbolAddress, once per device with
// that device current, and only that address is passed to kernels.
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

hipError_t hash_scratch(hipStream_t stream, void **ptr) {
  static std::mutex mu;
  static void *known[64];
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lk(mu);
  if (known[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    // the scan's ticket counter must start at zero; each call leaves it so
    e = launch_hash_scan_reset(static_cast<uint8_t *>(p) + kScratchState, stream);
    if (e != hipSuccess) return e;
    known[dev] = p;
  }
  *ptr = known[dev];
  return hipSuccess;
}

}  // namespace ea
