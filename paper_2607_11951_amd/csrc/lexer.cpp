// lexer.cpp -- the union lexer DFA over every declared terminal.
//
// Each terminal's regex becomes a position (Glushkov) automaton; the union of
// all of them is determinized by subset construction over byte classes,
// minimized (partition refinement), and annotated with per-state accept
// lists in priority order and the set of terminals still reachable ("live",
// used by the trailing-lexeme test of Definition 2).  The lexer must be
// gap-free: after a state accepts, every live state reachable from it accepts
// too, so the last accept of a pending lexeme is always its full length.
#include <algorithm>
#include <bitset>
#include <map>
#include <numeric>
#include <set>

#include "host.h"

namespace grid {
namespace {

struct RNode {
  enum Kind { SET, CAT, ALT, STAR, PLUS, OPT } kind = SET;
  std::bitset<256> set;
  int a = -1, b = -1;
};

struct RegexParser {
  const std::string& src;
  const std::string& name;
  size_t i = 0;
  std::vector<RNode>& nodes;
  RegexParser(const std::string& s, const std::string& n, std::vector<RNode>& out)
      : src(s), name(n), nodes(out) {}

  [[noreturn]] void fail(const std::string& m) {
    throw Error(GRID_E_GRAMMAR_SYNTAX, "regex of " + name + ": " + m);
  }
  int make(RNode n) {
    nodes.push_back(n);
    return (int)nodes.size() - 1;
  }
  int parse_byte_escape() {  // at '\\'
    if (i + 1 >= src.size()) fail("dangling escape");
    char e = src[i + 1];
    i += 2;
    switch (e) {
      case 'n': return '\n';
      case 't': return '\t';
      case 'r': return '\r';
      case 'x': {
        auto hv = [&](char ch) -> int {
          if (ch >= '0' && ch <= '9') return ch - '0';
          if (ch >= 'a' && ch <= 'f') return ch - 'a' + 10;
          if (ch >= 'A' && ch <= 'F') return ch - 'A' + 10;
          fail("bad hex digit");
        };
        if (i + 1 >= src.size()) fail("short \\x escape");
        int v = hv(src[i]) * 16 + hv(src[i + 1]);
        i += 2;
        return v;
      }
      default:
        if (isalnum((unsigned char)e)) fail(std::string("unknown escape \\") + e);
        return (unsigned char)e;
    }
  }
  int parse_alt() {
    int left = parse_cat();
    while (i < src.size() && src[i] == '|') {
      ++i;
      int right = parse_cat();
      RNode n;
      n.kind = RNode::ALT;
      n.a = left;
      n.b = right;
      left = make(n);
    }
    return left;
  }
  int parse_cat() {
    int acc = -1;
    while (i < src.size() && src[i] != '|' && src[i] != ')') {
      int r = parse_rep();
      if (acc < 0) {
        acc = r;
      } else {
        RNode n;
        n.kind = RNode::CAT;
        n.a = acc;
        n.b = r;
        acc = make(n);
      }
    }
    if (acc < 0) fail("empty alternative");
    return acc;
  }
  int parse_rep() {
    int x = parse_atom();
    while (i < src.size() && (src[i] == '*' || src[i] == '+' || src[i] == '?')) {
      RNode n;
      n.kind = src[i] == '*' ? RNode::STAR : (src[i] == '+' ? RNode::PLUS : RNode::OPT);
      n.a = x;
      ++i;
      x = make(n);
    }
    return x;
  }
  int parse_atom() {
    if (i >= src.size()) fail("unexpected end");
    char ch = src[i];
    RNode n;
    if (ch == '(') {
      ++i;
      int inner = parse_alt();
      if (i >= src.size() || src[i] != ')') fail("missing ')'");
      ++i;
      return inner;
    }
    if (ch == '.') {
      ++i;
      n.set.set();
      return make(n);
    }
    if (ch == '[') {
      ++i;
      bool negate = i < src.size() && src[i] == '^';
      if (negate) ++i;
      bool any = false;
      while (i < src.size() && (src[i] != ']' || !any)) {
        any = true;
        int lo = src[i] == '\\' ? parse_byte_escape() : (unsigned char)src[i++];
        int hi = lo;
        if (i + 1 < src.size() && src[i] == '-' && src[i + 1] != ']') {
          ++i;
          hi = src[i] == '\\' ? parse_byte_escape() : (unsigned char)src[i++];
        }
        if (hi < lo) fail("reversed range");
        for (int v = lo; v <= hi; ++v) n.set.set(v);
      }
      if (i >= src.size()) fail("unterminated class");
      ++i;
      if (negate) n.set.flip();
      if (n.set.none()) fail("empty class");
      return make(n);
    }
    if (ch == ')' || ch == '*' || ch == '+' || ch == '?' || ch == '|') fail("misplaced operator");
    int v = ch == '\\' ? parse_byte_escape() : (unsigned char)src[i++];
    n.set.set(v);
    return make(n);
  }
};

// Glushkov functions over the AST
struct Glushkov {
  const std::vector<RNode>& nodes;
  std::vector<int> leaf_pos;                 // node -> position or -1
  std::vector<std::bitset<256>> pos_set;     // position -> bytes
  std::vector<int> pos_term;
  std::vector<std::vector<int>> follow;
  explicit Glushkov(const std::vector<RNode>& n) : nodes(n), leaf_pos(n.size(), -1) {}

  struct Info {
    bool nullable;
    std::vector<int> first, last;
  };
  static std::vector<int> unite(const std::vector<int>& x, const std::vector<int>& y) {
    std::vector<int> out;
    std::set_union(x.begin(), x.end(), y.begin(), y.end(), std::back_inserter(out));
    return out;
  }
  void add_follow(const std::vector<int>& from, const std::vector<int>& to) {
    for (int p : from) follow[p] = unite(follow[p], to);
  }
  Info walk(int id, int term) {
    const RNode& n = nodes[id];
    switch (n.kind) {
      case RNode::SET: {
        int p = (int)pos_set.size();
        pos_set.push_back(n.set);
        pos_term.push_back(term);
        follow.emplace_back();
        leaf_pos[id] = p;
        return {false, {p}, {p}};
      }
      case RNode::CAT: {
        Info x = walk(n.a, term), y = walk(n.b, term);
        add_follow(x.last, y.first);
        Info r;
        r.nullable = x.nullable && y.nullable;
        r.first = x.nullable ? unite(x.first, y.first) : x.first;
        r.last = y.nullable ? unite(x.last, y.last) : y.last;
        return r;
      }
      case RNode::ALT: {
        Info x = walk(n.a, term), y = walk(n.b, term);
        return {x.nullable || y.nullable, unite(x.first, y.first), unite(x.last, y.last)};
      }
      case RNode::STAR:
      case RNode::PLUS: {
        Info x = walk(n.a, term);
        add_follow(x.last, x.first);
        return {n.kind == RNode::STAR || x.nullable, x.first, x.last};
      }
      case RNode::OPT: {
        Info x = walk(n.a, term);
        return {true, x.first, x.last};
      }
    }
    return {};
  }
};

}  // namespace

LexerDfa build_lexer(const GrammarText& g) {
  const int T = (int)g.terminals.size();
  std::vector<RNode> nodes;
  std::vector<int> roots(T);
  for (int t = 0; t < T; ++t) {
    const Terminal& term = g.terminals[t];
    if (term.regex) {
      RegexParser rp(term.source, term.name, nodes);
      roots[t] = rp.parse_alt();
      if (rp.i != term.source.size()) rp.fail("unbalanced ')'");
    } else {
      int acc = -1;
      for (unsigned char ch : term.source) {
        RNode leaf;
        leaf.set.set(ch);
        if (term.nocase && isalpha(ch)) leaf.set.set((unsigned char)(ch ^ 0x20));
        nodes.push_back(leaf);
        int id = (int)nodes.size() - 1;
        if (acc < 0) {
          acc = id;
        } else {
          RNode c;
          c.kind = RNode::CAT;
          c.a = acc;
          c.b = id;
          nodes.push_back(c);
          acc = (int)nodes.size() - 1;
        }
      }
      roots[t] = acc;
    }
  }
  Glushkov gk(nodes);
  std::vector<int> initial;              // first positions of every terminal
  std::vector<std::vector<int>> accepts_of_pos;
  std::vector<char> is_last;
  {
    std::vector<std::vector<int>> lasts(T);
    for (int t = 0; t < T; ++t) {
      Glushkov::Info inf = gk.walk(roots[t], t);
      if (inf.nullable)
        throw Error(GRID_E_GRAMMAR_SYNTAX, "token " + g.terminals[t].name + " matches the empty string");
      initial = Glushkov::unite(initial, inf.first);
      lasts[t] = inf.last;
    }
    is_last.assign(gk.pos_set.size(), 0);
    for (int t = 0; t < T; ++t)
      for (int p : lasts[t]) is_last[p] = 1;
  }
  const int P = (int)gk.pos_set.size();

  // byte classes: refine 0..255 by every position's byte set
  std::vector<int> cls(256, 0);
  {
    int ncls = 1;
    for (int p = 0; p < P; ++p) {
      std::map<std::pair<int, int>, int> remap;
      int next_id = 0;
      for (int b = 0; b < 256; ++b) {
        auto key = std::make_pair(cls[b], (int)gk.pos_set[p].test(b));
        auto it = remap.find(key);
        if (it == remap.end()) it = remap.emplace(key, next_id++).first;
        cls[b] = it->second;
      }
      ncls = next_id;
    }
    (void)ncls;
  }
  int C0 = *std::max_element(cls.begin(), cls.end()) + 1;
  std::vector<int> rep(C0, -1);
  for (int b = 0; b < 256; ++b)
    if (rep[cls[b]] < 0) rep[cls[b]] = b;

  // subset construction; state 0 = empty set (dead), state 1 = initial
  std::vector<std::vector<int>> states;
  std::map<std::vector<int>, int> index;
  auto intern = [&](const std::vector<int>& s) {
    auto it = index.find(s);
    if (it != index.end()) return it->second;
    int id = (int)states.size();
    index.emplace(s, id);
    states.push_back(s);
    return id;
  };
  intern({});
  intern({-1});  // marker for the initial state
  std::vector<std::vector<int>> trans;
  for (size_t s = 0; s < states.size(); ++s) {
    std::vector<int> row(C0, 0);
    if (s != 0) {
      for (int c = 0; c < C0; ++c) {
        int b = rep[c];
        std::vector<int> nxt;
        const std::vector<int> cur = states[s];
        for (int p : cur) {
          const std::vector<int>& succ = p < 0 ? initial : gk.follow[p];
          for (int q : succ)
            if (gk.pos_set[q].test(b)) nxt.push_back(q);
        }
        std::sort(nxt.begin(), nxt.end());
        nxt.erase(std::unique(nxt.begin(), nxt.end()), nxt.end());
        row[c] = intern(nxt);
      }
    }
    trans.push_back(row);
  }
  const int S0 = (int)states.size();
  std::vector<std::vector<int>> acc0(S0);
  for (int s = 0; s < S0; ++s) {
    std::set<int> a;
    for (int p : states[s])
      if (p >= 0 && is_last[p]) a.insert(gk.pos_term[p]);
    acc0[s].assign(a.begin(), a.end());
  }

  // minimization by partition refinement (Moore): blocks split by accept sets,
  // then by the blocks of their successors until stable
  std::vector<int> block(S0);
  {
    std::map<std::vector<int>, int> sig;
    for (int s = 0; s < S0; ++s) {
      auto it = sig.find(acc0[s]);
      if (it == sig.end()) it = sig.emplace(acc0[s], (int)sig.size()).first;
      block[s] = it->second;
    }
    for (int nblocks = (int)sig.size();;) {
      std::map<std::vector<int>, int> sig2;
      std::vector<int> nb(S0);
      for (int s = 0; s < S0; ++s) {
        std::vector<int> key;
        key.reserve(C0 + 1);
        key.push_back(block[s]);
        for (int c = 0; c < C0; ++c) key.push_back(block[trans[s][c]]);
        auto it = sig2.find(key);
        if (it == sig2.end()) it = sig2.emplace(key, (int)sig2.size()).first;
        nb[s] = it->second;
      }
      block.swap(nb);
      if ((int)sig2.size() == nblocks) break;
      nblocks = (int)sig2.size();
    }
  }
  // renumber: dead block -> 0, start block -> 1, others in order of first use
  const int nblk = *std::max_element(block.begin(), block.end()) + 1;
  std::vector<int> newid(nblk, -1);
  newid[block[0]] = kDead;
  if (block[1] == block[0]) throw Error(GRID_E_GRAMMAR_SYNTAX, "lexer accepts nothing");
  newid[block[1]] = kStart;
  int S = 2;
  for (int s = 0; s < S0; ++s)
    if (newid[block[s]] < 0) newid[block[s]] = S++;
  std::vector<int> repr(S, -1);
  for (int s = 0; s < S0; ++s)
    if (repr[newid[block[s]]] < 0) repr[newid[block[s]]] = s;

  // merge byte classes whose columns agree in the minimized automaton
  std::vector<int> colid(C0);
  int C = 0;
  {
    std::map<std::vector<int>, int> cols;
    for (int c = 0; c < C0; ++c) {
      std::vector<int> col(S);
      for (int q = 0; q < S; ++q) col[q] = newid[block[trans[repr[q]][c]]];
      auto it = cols.find(col);
      if (it == cols.end()) it = cols.emplace(col, C++).first;
      colid[c] = it->second;
    }
  }
  if (S > 0xFFFF) throw Error(GRID_E_CAPACITY, "lexer DFA has more than 65535 states");

  LexerDfa d;
  d.S = S;
  d.C = C;
  for (int b = 0; b < 256; ++b) d.byte_class[b] = (uint8_t)colid[cls[b]];
  d.next.assign((size_t)S * C, 0);
  d.dense.assign((size_t)S * 256, 0);
  for (int q = 0; q < S; ++q) {
    for (int c = 0; c < C0; ++c)
      d.next[(size_t)q * C + colid[c]] = (uint16_t)newid[block[trans[repr[q]][c]]];
    for (int b = 0; b < 256; ++b) d.dense[(size_t)q * 256 + b] = d.next[(size_t)q * C + d.byte_class[b]];
  }
  d.accepting.assign(S, 0);
  d.accept_off.assign(S + 1, 0);
  std::vector<std::vector<int>> acc(S);
  for (int q = 0; q < S; ++q) {
    acc[q] = acc0[repr[q]];
    std::sort(acc[q].begin(), acc[q].end(), [&](int x, int y) {
      const Terminal &tx = g.terminals[x], &ty = g.terminals[y];
      return tx.priority != ty.priority ? tx.priority > ty.priority : x < y;
    });
    d.accepting[q] = !acc[q].empty();
    d.accept_off[q + 1] = d.accept_off[q] + (uint32_t)acc[q].size();
    for (int t : acc[q]) d.accept_list.push_back((uint8_t)t);
  }
  // live terminals: least fixpoint of live(q) = acc(q) u live(successors)
  d.live.assign((size_t)S * kTermWords, 0);
  for (int q = 0; q < S; ++q)
    for (int t : acc[q]) d.live[(size_t)q * kTermWords + (t >> 5)] |= 1u << (t & 31);
  for (bool changed = true; changed;) {
    changed = false;
    for (int q = 1; q < S; ++q)
      for (int c = 0; c < C; ++c) {
        int r = d.next[(size_t)q * C + c];
        for (int w = 0; w < kTermWords; ++w) {
          uint32_t add = d.live[(size_t)r * kTermWords + w] & ~d.live[(size_t)q * kTermWords + w];
          if (add) {
            d.live[(size_t)q * kTermWords + w] |= add;
            changed = true;
          }
        }
      }
  }
  // gap-freedom
  for (int p = 1; p < S; ++p) {
    if (!d.accepting[p]) continue;
    std::vector<char> seen(S, 0);
    std::vector<int> stack{p};
    seen[p] = 1;
    while (!stack.empty()) {
      int u = stack.back();
      stack.pop_back();
      if (!d.accepting[u]) {
        std::string who;
        for (int t = 0; t < T; ++t)
          if (d.live[(size_t)u * kTermWords + (t >> 5)] >> (t & 31) & 1) who += g.terminals[t].name + " ";
        throw Error(GRID_E_LEXER_GAP,
                    "lexer gap: a non-accepting live state follows an accepting one (live: " + who + ")");
      }
      for (int c = 0; c < C; ++c) {
        int v = d.next[(size_t)u * C + c];
        if (v != kDead && !seen[v]) {
          seen[v] = 1;
          stack.push_back(v);
        }
      }
    }
  }
  return d;
}

}  // namespace grid
