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
// (state, nonterminal), 2^hbits slots of (key, target), linear probing, key 0
// empty.
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

// Words of one compact LR state record for terminal sets of tw words: shift
// bits, main reduce bits, main production, extra groups; padded to 16 bytes.
GRID_HD constexpr int parse_record_words(int tw) { return (2 * tw + 2 + 3) & ~3; }

GRID_HD uint32_t lexp_hash(uint32_t lo, uint32_t hi, uint32_t len) {
  uint32_t h = lo * 0x9E3779B1u ^ hi * 0x85EBCA77u ^ len * 0xC2B2AE3Du;
  h ^= h >> 15;
  h *= 0x2C1B3C6Du;
  return h ^ (h >> 12);
}

// Scan summary word of (lexer DFA state q, spelling u): how maximal munch
// segments the bytes of u when the scan resumes in q.  Bits 0-8: the DFA
// state after the last byte; 9-17: the state in which the first lexeme ended;
// 18-25: the index of the byte that ended it; 26-27: the number of lexeme ends
// inside u (2 = two or more); bit 28: the lexer alone rejects u (a lexeme
// ends in a state that accepts nothing, or a byte starts no lexeme).  The
// table exists when the DFA has at most 512 states.
constexpr uint32_t kScanMaxStates = 512;
constexpr uint32_t kScanReject = 1u << 28;
GRID_HD uint32_t scan_word(uint32_t q_end, uint32_t q_first, uint32_t p_first, uint32_t ends) {
  return q_end | q_first << 9 | p_first << 18 | ends << 26;
}
GRID_HD uint32_t scan_q_end(uint32_t w) { return w & 0x1FFu; }
GRID_HD uint32_t scan_q_first(uint32_t w) { return (w >> 9) & 0x1FFu; }
GRID_HD uint32_t scan_p_first(uint32_t w) { return (w >> 18) & 0xFFu; }
GRID_HD uint32_t scan_ends(uint32_t w) { return (w >> 26) & 3u; }

// Per-slot record (8 u32): flags base, hash base (entries), hash mask,
// restricted-category mask, node count, prefix-table base (entries),
// prefix-table mask, 1 reserved.
constexpr int kSlotWords = 8;

}  // namespace grid
