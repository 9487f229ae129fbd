// host.h -- host-side artifacts of a compiled grammar + vocabulary + lexicons.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <mutex>
#include <stdexcept>
#include <string>
#include <vector>

#include "../../include/grid.h"
#include "lexhash.h"

namespace grid {

constexpr int kMaxTerminals = 255;     // terminal ids fit a byte; column T is end of input
constexpr int kTermWords = 8;          // 256-bit terminal sets
constexpr int kMaxCategories = 8;
constexpr uint32_t kNoLex = 0xFFFFFFFFu;
constexpr uint16_t kActShift = 0x4000, kActReduce = 0x8000, kActAccept = 0xC000;
constexpr uint16_t kNoGoto = 0xFFFF;
constexpr uint32_t kSymNonterminal = 0x10000u, kNoSymbol = 0xFFFFFFFFu;
constexpr int kDead = 0, kStart = 1;   // lexer DFA state numbering

struct Error : std::runtime_error {
  int code;
  Error(int c, const std::string& m) : std::runtime_error(m), code(c) {}
};

// ---- grammar as read from text
struct Terminal {
  std::string name;
  bool regex = false;       // else literal
  std::string source;       // regex text or literal bytes
  bool nocase = false, ignored = false, category = false;
  int priority = 0;
};

struct Production {
  int lhs = 0;               // nonterminal index
  std::vector<int> rhs;      // >= 0 terminal id, < 0: nonterminal ~index
  std::string label;
};

struct GrammarText {
  std::vector<Terminal> terminals;
  std::vector<std::string> nonterminals;
  std::vector<Production> productions;
  int start = -1;
};

GrammarText parse_grammar(const std::string& text);

// per-lane parser overlay capacity of the mask kernels
int overlay_capacity();

// ---- lexer DFA (state 0 dead, 1 start)
struct LexerDfa {
  int S = 0, C = 0;
  uint8_t byte_class[256] = {};
  std::vector<uint16_t> next;          // [S*C]
  std::vector<uint16_t> dense;         // [S*256]
  std::vector<uint8_t> accepting;      // [S]
  std::vector<uint32_t> accept_off;    // [S+1]
  std::vector<uint8_t> accept_list;    // priority order (priority desc, id asc)
  std::vector<uint32_t> live;          // [S*kTermWords]
  uint16_t step(int q, uint8_t b) const { return next[(size_t)q * C + byte_class[b]]; }
};

LexerDfa build_lexer(const GrammarText& g);

// ---- LALR(1) parser over the projected, reduced grammar
struct Parser {
  int T = 0;                  // terminals; column T = end of input
  int N = 0;                  // nonterminals (renumbered after reduction)
  int n_states = 0;
  std::vector<uint16_t> action;   // [n_states*(T+1)]
  std::vector<uint16_t> go;       // [n_states*N]
  std::vector<uint16_t> go_skip;  // [n_states*N]: GOTO with transitions into unit states redirected
  std::vector<uint32_t> prod;     // lhs | len << 16
  std::vector<uint8_t> term_used; // terminal appears in the reduced grammar
  // compact form for set simulation (TW = words per terminal set incl. end of
  // input, a power of two): per state, parse_record_words(TW) words
  // [shift bits TW][main reduce bits TW][main production][extra groups | offset << 8]
  // (productions as lhs | length << 16, 0xFFFFFFFF none)
  int tw = 0;
  std::vector<uint32_t> pstate;
  std::vector<uint32_t> predx;     // extra reduce groups: [production][bits TW]
  std::vector<uint16_t> pshift;    // shift targets per state, in terminal order (record word 2TW+2)
  // GOTO as an open-addressing hash of H (power of two) u32 pairs: key
  // (state << 16 | nonterminal) + 1 (0 empty), target
  std::vector<uint32_t> goto_hash;
  int goto_hbits = 0;
  // accessing symbol of each LR state: terminal id, or kSymNonterminal |
  // nonterminal index; kNoSymbol for the initial state
  std::vector<uint32_t> state_sym;
  // fewest terminals that finish one kernel item of each state (completion search)
  std::vector<uint16_t> complete_est;
  uint16_t act(int s, int t) const { return action[(size_t)s * (T + 1) + t]; }
  uint16_t gto(int s, int a) const { return go[(size_t)s * N + a]; }
};

Parser build_parser(const GrammarText& g, const std::vector<std::string>& drop);

// Host LR simulation of terminal t (the end of input is t = T) on the stack:
// its reduce chain, then the shift; with commit the stack is changed, else a
// copy is used.  kSimShift, kSimAccept or kSimError.
enum SimResult { kSimError = 0, kSimShift = 1, kSimAccept = 2 };
int lr_simulate(const Parser& P, std::vector<uint16_t>& stack, int t, bool commit);

// ---- vocabulary
struct VocabArtifacts {
  int V = 0;
  std::vector<uint32_t> spell_off;   // [U+1]
  std::vector<uint8_t> spell_bytes;  // + padding
  std::vector<uint32_t> spell_rec;   // [U][4]: head lo, head hi, id | multi << 31, length | chunk << 8
  std::vector<uint8_t> spell_tail;   // bytes 8.. per spelling, 16-byte aligned chunks
  std::vector<uint16_t> sub_range;   // per 64 spellings: lowest | highest first byte << 8
  std::vector<uint32_t> spell_of_id; // [V]: spelling index, 0xFFFFFFFF none
  std::vector<uint8_t> id_first;     // [V]: first byte of the spelling, 0 none
  std::vector<uint32_t> id_head;     // [V]: first byte | second byte << 8 | 0x10000 if it has one
  std::vector<uint32_t> alias_off;   // [U+1]
  std::vector<int32_t> alias_ids;
  std::vector<uint32_t> level_off;   // [Lmax+2]
  std::vector<uint32_t> trie_nodes;  // [n*2]
  int max_len = 0;
  bool byte_complete = false;
  int eos_id = -1;
};

VocabArtifacts build_vocab(const uint8_t* bytes, const uint64_t* off, int V, const int32_t* specials,
                           int n_special, int eos_id);

// lexeme-program classes per lexer state (lexhash.h)
struct ClassTables {
  std::vector<uint16_t> map;   // [S][V] local class of each token id
  std::vector<uint32_t> off;   // [S+1] first record of each state
  std::vector<uint32_t> rec;   // [classes][4]
  uint32_t max_classes = 0;    // largest class count of one state
};
ClassTables build_class_tables(const LexerDfa& dfa, const VocabArtifacts& va);

// ---- lexicon slots
struct LexiconStore {
  std::vector<uint16_t> flags;     // all slots' nodes
  std::vector<uint32_t> child_bits;  // all slots' nodes: bitmap of the bytes with a child (8 u32 each)
  std::vector<uint32_t> hash;      // all slots' entries (2 u32 each)
  std::vector<uint32_t> prefix;    // all slots' prefix-table entries (4 u32 each)
  std::vector<uint32_t> stride;    // all slots' stride-table entries (8 u32 each)
  std::vector<uint32_t> token;     // all slots' token flags ([V] u32 each)
  std::vector<uint8_t> toksum;     // all slots' token-flag summaries ([V] u8 each: nonzero bytes of token)
  std::vector<uint32_t> slots;     // kSlotWords u32 per slot
  int n_slots = 0;
  // host-side lookup helpers
  uint32_t child(int slot, uint32_t node, uint8_t b) const;
  uint16_t node_flags(int slot, uint32_t node) const;
  uint32_t restricted(int slot) const { return slots[(size_t)slot * kSlotWords + 3]; }
  // the shortest words of each category of each slot (completion spellings)
  std::vector<std::vector<std::string>> shortest;  // [slot * kMaxCategories + category]
  const std::vector<std::string>& short_words(int slot, int cat) const {
    static const std::vector<std::string> none;
    const size_t i = (size_t)slot * kMaxCategories + (size_t)cat;
    return cat >= 0 && i < shortest.size() ? shortest[i] : none;
  }
};

void add_lexicon(LexiconStore& store, const LexerDfa& dfa, const GrammarText& g, const VocabArtifacts& va,
                 const std::vector<int>& term_cat,
                 const std::vector<std::pair<std::string, std::vector<std::string>>>& cats);

}  // namespace grid

struct grid_compiled {
  grid::GrammarText gram;
  grid::LexerDfa dfa;
  grid::Parser parser;
  grid::VocabArtifacts vocab;
  grid::LexiconStore lex;
  grid::ClassTables classes;          // lexeme-program classes
  uint32_t fingerprint = 0;           // of the lexer, parser and vocabulary (mask-cache entries)
  uint32_t family_fp = 0;             // of the lexer and vocabulary only (shared by every role)
  std::vector<int> term_cat;          // category index per terminal or -1
  std::vector<uint32_t> term_info;    // device word per terminal
  std::vector<int> cat_term;          // terminal id per category index
  std::mutex aux_mu;                  // guards the tables below, built on first use
  std::shared_ptr<void> writer;       // completion-writer tables (complete.cpp)
  void* dev[GRID_ART_COUNT] = {};
  size_t dev_bytes[GRID_ART_COUNT] = {};
};
