// lexhash.h -- hash layouts shared by the host builders and the kernels.
//
// A schema lexicon (section 2, L3) is one byte trie holding every category's
// words; edges live in an open-addressing table keyed by (node, byte).  Key 0
// marks an empty entry; child 0xFFFFFFFF never occurs in the table.
//
// Every lexicon-trie node of depth 1..8 is also in a prefix table keyed
// exactly by its bytes (two little-endian words, zero padded) and length, so
// a lexeme of at most 8 bytes is looked up with one probe.
//
// The LR GOTO function lives in a third open-addressing table keyed by
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

GRID_HD uint32_t lexp_hash(uint32_t lo, uint32_t hi, uint32_t len) {
  uint32_t h = lo * 0x9E3779B1u ^ hi * 0x85EBCA77u ^ len * 0xC2B2AE3Du;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  return h ^ (h >> 12);
}

// Per-slot record (8 u32): flags base, hash base (entries), hash mask,
// restricted-category mask, node count, prefix-table base (entries),
// prefix-table mask, 1 reserved.
constexpr int kSlotWords = 8;

}  // namespace grid
