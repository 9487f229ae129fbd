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

// Stride table: every lexicon-trie node of depth d > 8, keyed by its
// ancestor at depth 8 * floor((d - 1) / 8) and its bytes below that ancestor
// (1..8, little-endian, zero padded), so a lexeme of up to 24 bytes is looked
// up with at most three probes.  Entry, 8 u32: ancestor node, bytes lo,
// bytes hi, length | flags << 16 (length 0 = empty), node, 0, 0, 0.
GRID_HD uint32_t lexs_hash(uint32_t anc, uint32_t lo, uint32_t hi, uint32_t len) {
  return lexp_hash(lo ^ anc * 0x27D4EB2Fu, hi + anc, len);
}

// Lexeme-program classes (verdict-equivalence classes of section 4.2, keyed
// by lexer state).  When the scan resumes in DFA state q, maximal munch cuts
// the bytes of a token into lexemes independently of the parser (munch length
// comes from the lexer alone); what the parser later decides depends only on
// the DFA states in which those lexemes end and the state after the last
// byte.  Tokens with equal programs from q form a class; CLASS_MAP[q][id] is
// the token's class index local to q, and the classes of q are the records
// CLASS_REC[CLASS_OFF[q] ...], four u32 each:
//   w0: ends (0..kClassEnds, kClassMore = more) | reject | first-byte-ends-lexeme
//   w1: state after the last byte | state where lexeme 0 ended << 16
//   w2: state where lexeme 1 ended | state where lexeme 2 ended << 16
//   w3: the byte indices that ended lexemes 0, 1, 2 (8 bits each, 0 for
//       missing ends): lexeme 0 is the pending bytes and the token's bytes
//       before its end, lexeme i the bytes between ends i-1 and i, and the
//       trailing lexeme the bytes after the last end (all of the token and
//       the pending bytes when there is none)
// Local class 0 of every state is "rejected by the lexer alone" (also special
// and empty tokens); local class 1 is "walk the bytes" (tokens of a state
// whose class count exceeds 65536).
constexpr int kClassEnds = 3;
constexpr uint32_t kClassMore = 4;
constexpr uint32_t kClassEndsMask = 7u;
constexpr uint32_t kClassReject = 1u << 3;
constexpr uint32_t kClassP0 = 1u << 4;
constexpr uint32_t kClassWalk = 1u << 5;
constexpr uint32_t kClassMaxLocal = 65536;

// Per-slot record (12 u32): flags base, hash base (entries), hash mask,
// restricted-category mask, node count, prefix-table base (entries),
// prefix-table mask, stride-table base (entries), stride-table mask, 3
// reserved.
constexpr int kSlotWords = 12;

}  // namespace grid
