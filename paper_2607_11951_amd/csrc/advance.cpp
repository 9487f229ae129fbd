// advance.cpp -- host advance: prefix bytes -> parser configuration.
//
// This is the per-token step 7 of section 6.1 run over a whole prefix: bytes
// go through the lexer DFA with maximal munch; when a byte kills the DFA the
// pending lexeme is emitted as the highest-priority candidate that the LALR
// parser can shift (or an ignored one) and that passes its category's lexicon;
// a shifted terminal runs its reduce chain on the stack.  The result is the
// configuration of Definition 1: the stack right after the last shift, the
// DFA state of the pending lexeme and its lexicon-trie node.  The prefix must
// be viable (Definition 2), i.e. the pending lexeme is live for an allowed or
// ignored terminal.
#include <cstring>

#include "host.h"
#include "lexhash.h"

namespace grid {

// Reduce chain for terminal t on a copy of the stack; with commit, the real
// stack is reduced and t shifted.
int lr_simulate(const Parser& P, std::vector<uint16_t>& stack, int t, bool commit) {
  std::vector<uint16_t> scratch;
  std::vector<uint16_t>& st = commit ? stack : (scratch = stack);
  for (int guard = 0; guard < 1 << 20; ++guard) {
    uint16_t a = P.act(st.back(), t);
    if (a == 0) return kSimError;
    if ((a & 0xC000) == kActShift) {
      if (commit) st.push_back((uint16_t)(a & 0x3FFF));
      return kSimShift;
    }
    if ((a & 0xC000) == kActAccept) return kSimAccept;
    uint32_t pr = P.prod[a & 0x3FFF];
    size_t len = pr >> 16;
    if (len >= st.size()) return kSimError;
    st.resize(st.size() - len);
    uint16_t g = P.gto(st.back(), (int)(pr & 0xFFFF));
    if (g == kNoGoto) return kSimError;
    st.push_back(g);
  }
  return kSimError;
}

}  // namespace grid

using namespace grid;

int host_config_from_prefix(const grid_compiled* g, int slot, const uint8_t* w, size_t n,
                            grid_config* cfg, std::vector<uint16_t>& stack) {
  const LexerDfa& D = g->dfa;
  const Parser& P = g->parser;
  const LexiconStore& L = g->lex;
  const uint32_t restricted = L.restricted(slot);
  auto ignored = [&](int t) { return (g->term_info[t] & 1u) != 0; };
  auto cat_of = [&](int t) { return g->term_cat[t]; };
  auto lex_word_ok = [&](int t, uint32_t node) {
    int c = cat_of(t);
    if (c < 0 || !(restricted >> c & 1)) return true;
    return (L.node_flags(slot, node) >> (8 + c) & 1) != 0;
  };
  auto lex_prefix_ok = [&](int t, uint32_t node) {
    int c = cat_of(t);
    if (c < 0 || !(restricted >> c & 1)) return true;
    return (L.node_flags(slot, node) >> c & 1) != 0;
  };
  auto allowed = [&](int t) { return ignored(t) || lr_simulate(P, stack, t, false) == 1; };

  stack.assign(1, 0);
  int q = kStart;
  uint32_t lex = 0;  // root of the slot's lexicon trie
  uint32_t rem = 0;
  for (size_t i = 0; i < n; ++i) {
    uint8_t b = w[i];
    int nq = D.step(q, b);
    if (nq != kDead) {
      q = nq;
      lex = L.child(slot, lex, b);
      ++rem;
      continue;
    }
    // b kills the pending lexeme: emit it
    if (rem == 0 || !D.accepting[q]) return GRID_E_NOT_VIABLE;
    int win = -1;
    for (uint32_t k = D.accept_off[q]; k < D.accept_off[q + 1]; ++k) {
      int t = D.accept_list[k];
      if (allowed(t) && lex_word_ok(t, lex)) {
        win = t;
        break;
      }
    }
    if (win < 0) return GRID_E_NOT_VIABLE;
    if (!ignored(win) && lr_simulate(P, stack, win, true) != 1) return GRID_E_NOT_VIABLE;
    q = D.step(kStart, b);
    if (q == kDead) return GRID_E_NOT_VIABLE;
    lex = L.child(slot, 0, b);
    rem = 1;
  }
  if (rem > 0) {  // Definition 2: the pending lexeme is live for an allowed or ignored terminal
    bool ok = false;
    for (int t = 0; t < P.T && !ok; ++t)
      if ((D.live[(size_t)q * kTermWords + (t >> 5)] >> (t & 31) & 1) && allowed(t) && lex_prefix_ok(t, lex))
        ok = true;
    if (!ok) return GRID_E_NOT_VIABLE;
  }
  cfg->stk_off = 0;
  cfg->stk_depth = (uint32_t)stack.size();
  cfg->lexnode = lex;
  cfg->q = (uint16_t)q;
  cfg->slot = (uint16_t)slot;
  cfg->flags = rem == 0 ? 1u : 0u;
  cfg->rem_len = rem;
  memset(cfg->rem_head, 0, sizeof cfg->rem_head);
  for (uint32_t k = 0; k < rem && k < 8; ++k) cfg->rem_head[k] = w[n - rem + k];
  return GRID_OK;
}
