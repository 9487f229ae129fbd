// lexhash.h -- hash layouts shared by the host builders and the kernels.
//
// A schema lexicon (section 2, L3) is one byte trie holding every category's
// words; edges live in an open-addressing table keyed by (node, byte).  Key 0
// marks an empty entry; child 0xFFFFFFFF never occurs in the table.
//
// The LR GOTO function lives in a second open-addressing table keyed by
// (state, nonterminal), 2^hbits slots, linear probing, key 0 empty.
#pragma once
#include <cstdint>

#if defined(__HIPCC__)
#define GRID_HD __host__ __device__ __forceinline__
#else
#define GRID_HD inline
#endif

namespace grid {

GRID_HD uint32_t lex_key(uint32_t node, uint32_t byte) { return node * 256u + byte + 1u; }

GRID_HD uint32_t lex_hash(uint32_t key) {
  uint32_t h = key * 0x9E3779B1u;
  return h ^ (h >> 15);
}

GRID_HD uint32_t goto_key(uint32_t state, uint32_t nonterminal) { return (state << 16 | nonterminal) + 1u; }

GRID_HD uint32_t goto_slot(uint32_t key, int hbits) { return (key * 0x9E3779B1u) >> (32 - hbits); }

// Per-slot record (8 u32): flags base, hash base (entries), hash mask,
// restricted-category mask, node count, 3 reserved.
constexpr int kSlotWords = 8;

}  // namespace grid
