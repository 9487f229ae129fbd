// rolling_hash.h -- rolling configuration hash of an LR stack (section 6.4,
// the audit chain's configuration hash): every stack node's hash is
//   H(node) = low64(BLAKE2b-128(H(parent) || u32(state) || u32(goto))),
//   H(root) = 0,
// so a push costs one hash of a 16-byte message and a pop costs nothing (the
// parent's hash is kept with the parent).  Here a node is a stack entry: its
// parent is the entry below it, the root is the bottom entry (the initial LR
// state), `goto` is the symbol on which the automaton entered the state
// (terminal id, or 0x10000 | nonterminal index), H(parent) is serialized as
// 8 little-endian bytes, the u32 fields little-endian, and low64 is the first
// 8 bytes of the 16-byte digest read little-endian.
//
// BLAKE2b follows its published definition (RFC 7693): 64-bit words, the
// SHA-512 initial vector, 12 rounds of the G mixing function with the
// message schedule sigma; parameter block for an unkeyed 16-byte digest.
#pragma once
#include <cstdint>

#if defined(__HIPCC__)
#define GRID_RH __host__ __device__ __forceinline__
#else
#define GRID_RH inline
#endif

namespace grid {

constexpr uint64_t kBlake2bIv[8] = {0x6A09E667F3BCC908ull, 0xBB67AE8584CAA73Bull, 0x3C6EF372FE94F82Bull,
                                    0xA54FF53A5F1D36F1ull, 0x510E527FADE682D1ull, 0x9B05688C2B3E6C1Full,
                                    0x1F83D9ABFB41BD6Bull, 0x5BE0CD19137E2179ull};

constexpr uint8_t kBlake2bSigma[10][16] = {
    {0, 1, 2, 3, 4, 5, 6, 7, 8, 9, 10, 11, 12, 13, 14, 15}, {14, 10, 4, 8, 9, 15, 13, 6, 1, 12, 0, 2, 11, 7, 5, 3},
    {11, 8, 12, 0, 5, 2, 15, 13, 10, 14, 3, 6, 7, 1, 9, 4}, {7, 9, 3, 1, 13, 12, 11, 14, 2, 6, 5, 10, 4, 0, 15, 8},
    {9, 0, 5, 7, 2, 4, 10, 15, 14, 1, 11, 12, 6, 8, 3, 13}, {2, 12, 6, 10, 0, 11, 8, 3, 4, 13, 7, 5, 15, 14, 1, 9},
    {12, 5, 1, 15, 14, 13, 4, 10, 0, 7, 6, 3, 9, 2, 8, 11}, {13, 11, 7, 14, 12, 1, 3, 9, 5, 0, 15, 4, 8, 6, 2, 10},
    {6, 15, 14, 9, 11, 3, 0, 8, 12, 2, 13, 7, 1, 4, 10, 5}, {10, 2, 8, 4, 7, 6, 1, 5, 15, 11, 9, 14, 3, 12, 13, 0}};

GRID_RH uint64_t rotr64(uint64_t x, int n) { return (x >> n) | (x << (64 - n)); }

GRID_RH void blake2b_g(uint64_t* v, int a, int b, int c, int d, uint64_t x, uint64_t y) {
  v[a] = v[a] + v[b] + x;
  v[d] = rotr64(v[d] ^ v[a], 32);
  v[c] = v[c] + v[d];
  v[b] = rotr64(v[b] ^ v[c], 24);
  v[a] = v[a] + v[b] + y;
  v[d] = rotr64(v[d] ^ v[a], 16);
  v[c] = v[c] + v[d];
  v[b] = rotr64(v[b] ^ v[c], 63);
}

// The first 8 bytes (little-endian) of BLAKE2b-128 of the 16-byte message
// m0 || m1 (each 8 bytes little-endian): one final block, counter 16.
GRID_RH uint64_t blake2b128_low64_16(uint64_t m0, uint64_t m1) {
  uint64_t h[8], v[16], m[16];
  for (int i = 0; i < 8; ++i) h[i] = kBlake2bIv[i];
  h[0] ^= 0x01010000ull ^ 16ull;  // digest length 16, no key, fanout 1, depth 1
  for (int i = 0; i < 16; ++i) m[i] = 0;
  m[0] = m0;
  m[1] = m1;
  for (int i = 0; i < 8; ++i) {
    v[i] = h[i];
    v[i + 8] = kBlake2bIv[i];
  }
  v[12] ^= 16ull;  // bytes hashed so far (low word of the counter)
  v[14] = ~v[14];  // the final block
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
#endif
  for (int r = 0; r < 12; ++r) {
    const uint8_t* s = kBlake2bSigma[r % 10];
    blake2b_g(v, 0, 4, 8, 12, m[s[0]], m[s[1]]);
    blake2b_g(v, 1, 5, 9, 13, m[s[2]], m[s[3]]);
    blake2b_g(v, 2, 6, 10, 14, m[s[4]], m[s[5]]);
    blake2b_g(v, 3, 7, 11, 15, m[s[6]], m[s[7]]);
    blake2b_g(v, 0, 5, 10, 15, m[s[8]], m[s[9]]);
    blake2b_g(v, 1, 6, 11, 12, m[s[10]], m[s[11]]);
    blake2b_g(v, 2, 7, 8, 13, m[s[12]], m[s[13]]);
    blake2b_g(v, 3, 4, 9, 14, m[s[14]], m[s[15]]);
  }
  return h[0] ^ v[0] ^ v[8];
}

// H of a stack node from its parent's hash, its LR state and the symbol on
// which the state was entered.
GRID_RH uint64_t node_hash(uint64_t parent, uint32_t state, uint32_t sym) {
  return blake2b128_low64_16(parent, (uint64_t)state | (uint64_t)sym << 32);
}

}  // namespace grid
