// complete.cpp -- termination machinery on the host (section 5, Proposition 9
// mode 1; section 6.1 step 3): a legal completion of a viable prefix, counted
// in vocabulary tokens, which is also the prefix's reserve.
//
// The prefix's pending lexeme is finished first: the shortest byte extension
// after which the lexeme is accepted by a terminal the parser takes (or an
// ignored one) that wins contextual resolution and passes its category's
// lexicon, and after which a whitespace byte ends it.  Then a best-first
// search over terminal sequences runs on the LR stack: a move shifts one
// terminal the parser can take next, costing the tokens of a separator and of
// the terminal's spelling in that context (the shortest spelling that wins
// resolution there: the literal text, a shortest string of the terminal's
// regex, or a shortest word of its category in the row's schema lexicon); the
// estimate of what is left is the sum, over the stack, of the fewest
// terminals that finish one kernel item of each state, at two tokens each.  A
// configuration whose end-of-input chain reaches ACCEPT is complete.  The
// bytes are tokenized by greedy longest match and the whole output is checked
// to be a sentence of the language before it is returned.
#include <algorithm>
#include <cstring>
#include <mutex>
#include <queue>
#include <string>
#include <unordered_map>
#include <unordered_set>

#include "host.h"
#include "lexhash.h"

int host_config_from_prefix(const grid_compiled* g, int slot, const uint8_t* w, size_t n, grid_config* cfg,
                            std::vector<uint16_t>& stack);

namespace grid {
int fail(int code, const std::string& msg);
void clear_error();
}  // namespace grid

using namespace grid;

namespace {

// Per-handle tables the writer builds on first use.
struct WriterTables {
  std::vector<std::vector<std::string>> spell;    // per terminal: candidate spellings, shortest first
  std::unordered_map<std::string, int32_t> ids;   // spelling -> first token id
  std::vector<uint8_t> seps;                      // whitespace bytes that start an ignored lexeme
};

const WriterTables& writer_tables(const grid_compiled* gc) {
  grid_compiled* g = const_cast<grid_compiled*>(gc);  // only the lazily built tables change
  std::lock_guard<std::mutex> lock(g->aux_mu);
  if (g->writer) return *static_cast<const WriterTables*>(g->writer.get());
  auto holder = std::make_shared<WriterTables>();
  WriterTables& W = *holder;
  const LexerDfa& D = g->dfa;
  const int T = g->parser.T;
  W.spell.assign(T, {});
  // literal terminals spell themselves; every terminal also gets the
  // shortest strings reaching each DFA state that accepts it
  for (int t = 0; t < T; ++t)
    if (!g->gram.terminals[t].regex) W.spell[t].push_back(g->gram.terminals[t].source);
  std::vector<std::string> path(D.S);
  std::vector<char> seen(D.S, 0);
  std::vector<int> order{kStart};
  seen[kStart] = 1;
  for (size_t h = 0; h < order.size(); ++h) {
    const int q = order[h];
    for (int b = 0; b < 256; ++b) {
      const int nq = D.step(q, (uint8_t)b);
      if (nq == kDead || seen[nq]) continue;
      seen[nq] = 1;
      path[nq] = path[q] + (char)b;
      order.push_back(nq);
    }
  }
  for (int q : order)
    for (uint32_t k = D.accept_off[q]; k < D.accept_off[q + 1]; ++k) {
      const int t = D.accept_list[k];
      if (W.spell[t].size() < 6 && std::find(W.spell[t].begin(), W.spell[t].end(), path[q]) == W.spell[t].end())
        W.spell[t].push_back(path[q]);
    }
  for (auto& v : W.spell)
    std::stable_sort(v.begin(), v.end(), [](const std::string& a, const std::string& b) { return a.size() < b.size(); });
  const VocabArtifacts& va = g->vocab;
  for (size_t u = 0; u + 1 < va.spell_off.size(); ++u) {
    const std::string sp((const char*)va.spell_bytes.data() + va.spell_off[u], va.spell_off[u + 1] - va.spell_off[u]);
    W.ids.emplace(sp, va.alias_ids[va.alias_off[u]]);
  }
  for (uint8_t b : {(uint8_t)' ', (uint8_t)'\n', (uint8_t)'\t', (uint8_t)'\r'}) {
    const int q = D.step(kStart, b);
    if (q == kDead) continue;
    for (uint32_t k = D.accept_off[q]; k < D.accept_off[q + 1]; ++k)
      if (g->term_info[D.accept_list[k]] & 1u) {
        W.seps.push_back(b);
        break;
      }
  }
  g->writer = holder;
  return W;
}

struct Ctx {
  const grid_compiled* g;
  int slot;
  uint32_t restricted;
  bool ignored(int t) const { return (g->term_info[t] & 1u) != 0; }
  int cat(int t) const { return g->term_cat[t]; }
  bool is_restricted(int t) const { return cat(t) >= 0 && ((restricted >> cat(t)) & 1u); }
  uint32_t node_of(const std::string& s) const {
    uint32_t node = 0;
    for (unsigned char c : s) node = g->lex.child(slot, node, c);
    return node;
  }
  bool word_ok(int t, uint32_t node) const {
    return !is_restricted(t) || ((g->lex.node_flags(slot, node) >> (8 + cat(t))) & 1u);
  }
  // The winner of a lexeme ending in DFA state q with lexicon node `node` on
  // the stack: the first accept-list entry that is ignored or shifts and
  // passes its lexicon word test; -1 none.
  int winner(std::vector<uint16_t>& stack, int q, uint32_t node) const {
    const LexerDfa& D = g->dfa;
    for (uint32_t k = D.accept_off[q]; k < D.accept_off[q + 1]; ++k) {
      const int t = D.accept_list[k];
      if (!word_ok(t, node)) continue;
      if (ignored(t) || lr_simulate(g->parser, stack, t, false) == kSimShift) return t;
    }
    return -1;
  }
  int run(const std::string& s, int q = kStart) const {
    for (unsigned char c : s) {
      q = g->dfa.step(q, c);
      if (q == kDead) return kDead;
    }
    return q;
  }
};

// Greedy longest-match tokenization of bytes; false if some byte has no token.
bool tokenize(const WriterTables& W, int max_len, const std::string& bytes, std::vector<int32_t>& out) {
  size_t i = 0;
  while (i < bytes.size()) {
    bool found = false;
    for (size_t L = std::min<size_t>((size_t)max_len, bytes.size() - i); L >= 1; --L) {
      auto it = W.ids.find(bytes.substr(i, L));
      if (it != W.ids.end()) {
        out.push_back(it->second);
        i += L;
        found = true;
        break;
      }
    }
    if (!found) return false;
  }
  return true;
}

int count_tokens(const WriterTables& W, int max_len, const std::string& bytes) {
  std::vector<int32_t> t;
  return tokenize(W, max_len, bytes, t) ? (int)t.size() : 1 << 20;
}

}  // namespace

extern "C" int grid_complete(const grid_compiled* g, int32_t slot, const uint8_t* w, size_t n, int32_t max_tokens,
                             int32_t* out_tokens, int32_t* out_n) {
  clear_error();
  if (!g || !out_n || (n > 0 && !w) || max_tokens < 0 || (max_tokens > 0 && !out_tokens))
    return fail(GRID_E_ARG, "grid_complete: null argument");
  if (slot < 0 || slot >= g->lex.n_slots) return fail(GRID_E_ARG, "grid_complete: lexicon slot out of range");
  try {
    grid_config cfg;
    std::vector<uint16_t> stack;
    const int rc = host_config_from_prefix(g, slot, w, n, &cfg, stack);
    if (rc == GRID_E_NOT_VIABLE) return fail(rc, "grid_complete: the prefix is not viable");
    if (rc) return fail(rc, "grid_complete: configuration build failed");
    const WriterTables& W = writer_tables(g);
    if (W.seps.empty()) return fail(GRID_E_ARG, "grid_complete: the grammar has no ignored whitespace");
    const Ctx C{g, slot, g->lex.restricted(slot)};
    const LexerDfa& D = g->dfa;
    const Parser& P = g->parser;
    const int max_len = std::max(1, g->vocab.max_len);
    std::string tail;  // the bytes written after the prefix

    // 1. finish the pending lexeme: shortest extension e with a winner and a
    // separator byte that ends it
    if (!(cfg.flags & 1u)) {
      const std::string rem((const char*)w + n - cfg.rem_len, cfg.rem_len);
      struct Node {
        int q;
        std::string e;
      };
      std::vector<Node> frontier{{(int)cfg.q, ""}};
      std::unordered_set<uint64_t> seen{((uint64_t)cfg.q << 32) | cfg.lexnode};
      bool done = false;
      for (size_t h = 0; h < frontier.size() && !done && h < 200000; ++h) {
        const Node nd = frontier[h];
        if (D.accepting[nd.q]) {
          const uint32_t node = C.node_of(rem + nd.e);
          const int t = C.winner(stack, nd.q, node);
          int sep = -1;
          for (uint8_t b : W.seps)
            if (D.step(nd.q, b) == kDead) {
              sep = b;
              break;
            }
          // an ignored lexeme that the separator extends (whitespace) stays
          // ignored and is ended by the first byte of the next spelling
          if (sep < 0 && t >= 0 && C.ignored(t)) {
            const int q2 = D.step(nd.q, W.seps[0]);
            if (q2 != kDead && D.accepting[q2] && C.ignored(D.accept_list[D.accept_off[q2]])) sep = W.seps[0];
          }
          if (t >= 0 && sep >= 0) {
            if (!C.ignored(t)) lr_simulate(P, stack, t, true);
            tail = nd.e;
            if (sep != W.seps[0]) tail += (char)sep;  // the byte that ends the lexeme, when it differs
            done = true;
            break;
          }
        }
        if (nd.e.size() >= 64) continue;
        for (int b = 0; b < 256; ++b) {
          const int nq = D.step(nd.q, (uint8_t)b);
          if (nq == kDead) continue;
          const uint32_t node = C.restricted ? C.node_of(rem + nd.e + (char)b) : 0u;
          const uint64_t key = ((uint64_t)nq << 32) | node;
          if (!seen.insert(key).second) continue;
          frontier.push_back({nq, nd.e + (char)b});
        }
      }
      if (!done) return fail(GRID_E_CAPACITY, "grid_complete: the pending lexeme cannot be finished");
    }

    // 2. best-first search over terminal sequences on the stack
    const int T = P.T;
    auto estimate = [&](const std::vector<uint16_t>& st) {
      long e = 0;
      for (size_t i = 1; i < st.size(); ++i) e += P.complete_est[st[i]];
      return 2 * e;
    };
    struct SNode {
      std::vector<uint16_t> stack;
      std::string text;
      int cost;
    };
    struct Pri {
      long f;
      int idx;
      bool operator<(const Pri& o) const { return f > o.f || (f == o.f && idx > o.idx); }
    };
    std::vector<SNode> nodes{{stack, "", 0}};
    std::priority_queue<Pri> open;
    open.push({estimate(stack), 0});
    std::unordered_set<std::string> visited;
    int goal = -1;
    // the search is bounded by expansions and by the bytes its nodes hold
    // (every node keeps its whole stack: deep prefixes make nodes large)
    constexpr size_t kSearchBytes = size_t(256) << 20;
    size_t held = stack.size() * 2;
    for (int expansions = 0; !open.empty() && expansions < 60000 && held < kSearchBytes; ++expansions) {
      const int idx = open.top().idx;
      open.pop();
      std::vector<uint16_t> st = nodes[idx].stack;
      const std::string key((const char*)st.data(), st.size() * 2);
      if (!visited.insert(key).second) continue;
      if (lr_simulate(P, st, T, false) == kSimAccept) {
        goal = idx;
        break;
      }
      for (int t = 0; t < T; ++t) {
        if (C.ignored(t) || !P.term_used[t]) continue;
        if (lr_simulate(P, st, t, false) != kSimShift) continue;
        // the shortest spelling that wins resolution for t here
        std::string best;
        bool have = false;
        auto try_spell = [&](const std::string& s) {
          if (have && s.size() >= best.size()) return;
          const int q = C.run(s);
          if (q == kDead || !D.accepting[q]) return;
          std::vector<uint16_t> tmp = st;
          if (C.winner(tmp, q, C.node_of(s)) != t) return;
          best = s;
          have = true;
        };
        for (const std::string& s : W.spell[t]) try_spell(s);
        if (C.is_restricted(t))
          for (const std::string& s : g->lex.short_words(slot, C.cat(t))) try_spell(s);
        if (!have) continue;
        std::vector<uint16_t> child = st;
        lr_simulate(P, child, t, true);
        const std::string step = std::string(1, (char)W.seps[0]) + best;
        const int c = nodes[idx].cost + count_tokens(W, max_len, step);
        held += child.size() * 2 + nodes[idx].text.size() + step.size() + sizeof(SNode);
        nodes.push_back({std::move(child), nodes[idx].text + step, c});
        open.push({(long)c + estimate(nodes.back().stack), (int)nodes.size() - 1});
      }
    }
    if (goal < 0) return fail(GRID_E_CAPACITY, "grid_complete: no completion found within the search budget");
    tail += nodes[goal].text;

    // 3. tokens, and the whole output checked to be a sentence of L
    std::vector<int32_t> toks;
    if (!tokenize(W, max_len, tail, toks)) return fail(GRID_E_VOCAB, "grid_complete: a byte has no token");
    std::string all((const char*)w, n);
    all += tail;
    grid_config c2;
    std::vector<uint16_t> st2;
    if (host_config_from_prefix(g, slot, (const uint8_t*)all.data(), all.size(), &c2, st2) != GRID_OK)
      return fail(GRID_E_ARG, "grid_complete: the completion left the language (internal error)");
    bool member = false;
    if (c2.flags & 1u) {
      member = lr_simulate(P, st2, T, false) == kSimAccept;
    } else {
      const int t = C.winner(st2, c2.q, c2.lexnode);
      if (t >= 0) {
        if (!C.ignored(t)) lr_simulate(P, st2, t, true);
        member = lr_simulate(P, st2, T, false) == kSimAccept;
      }
    }
    if (!member) return fail(GRID_E_ARG, "grid_complete: the completion is not a sentence (internal error)");
    *out_n = (int32_t)toks.size();
    if ((int32_t)toks.size() > max_tokens)
      return fail(GRID_E_CAPACITY, "grid_complete: the completion needs " + std::to_string(toks.size()) + " tokens");
    if (!toks.empty()) std::memcpy(out_tokens, toks.data(), toks.size() * sizeof(int32_t));
    return GRID_OK;
  } catch (const std::exception& e) {
    return fail(GRID_E_ARG, e.what());
  }
}
