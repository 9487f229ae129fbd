// oracle.cpp -- CPU oracle for the exact grammar-constrained next-token mask.
//
// TEST INFRASTRUCTURE ONLY: loaded by the test suite, the package smoke check
// and the benchmark's CPU-baseline leg; never by the product path.  It shares
// no code with the HIP library.
//
// The mask is the plain definition (Definition 4, section 4.1):
//   M(w) = { t : w.bytes(t) in Prefix(L) }  u  { EOS iff w in L }.
// Prefix(L) membership is decided by the operational form of Definition 2
// (section 3.2): the incremental scan-and-parse of the bytes succeeds, and the
// trailing partial lexeme is live for a terminal that is allowed next or
// ignored.  L follows section 2: maximal munch over the union of all terminal
// regexes, where a forced emission carries every terminal accepting the
// longest match, category terminals keep only lexemes in their schema
// allow-list, and the highest-priority candidate the parser can accept (or an
// ignored one) wins; the role projection drops productions and then removes
// useless symbols.  Parser viability comes from an Earley recognizer: after a
// reduced grammar, a terminal is viable next iff some Earley item of the
// current set expects it.
//
// Readings where the paper is not explicit (also listed in the design notes):
//  * priorities are integers from the grammar file (literal tokens default 1,
//    regex tokens 0); ties go to the lower terminal id;
//  * no fallback to a shorter match when no candidate of the longest match
//    is viable: the input is rejected;
//  * lexicons only filter candidates at emission (whole-word membership) and
//    gate the trailing lexeme (prefix of some allowed word); munch length is
//    decided by the regexes alone;
//  * the lexer covers every declared terminal even when the projection made
//    it unreachable;
//  * end of input finalizes the pending lexeme like a killing byte.

#include "oracle.h"

#include <memory>
#include <algorithm>
#include <bitset>
#include <cctype>
#include <cstring>
#include <map>
#include <mutex>
#include <set>
#include <stdexcept>
#include <string>
#include <unordered_map>
#include <unordered_set>
#include <vector>

#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

using std::string;
using std::vector;

struct OracleError : std::runtime_error {
  using std::runtime_error::runtime_error;
};

// ------------------------------------------------------------------ grammar
struct TermDecl {
  string name;
  bool is_regex = false;
  string pattern;  // regex source or literal bytes
  bool nocase = false, ignore = false, category = false;
  int prio = 0;
};

struct Rule {
  int lhs;           // nonterminal index
  vector<int> rhs;   // symbol ids: terminal t -> t, nonterminal n -> T + n
  string label;
};

struct GrammarFile {
  vector<TermDecl> terms;
  vector<string> nonterms;
  vector<Rule> rules;
  string start;
};

static bool is_ident_char(char c) {
  return (c >= 'a' && c <= 'z') || (c >= 'A' && c <= 'Z') || (c >= '0' && c <= '9') || c == '_';
}

static int hexval(char c) {
  if (c >= '0' && c <= '9') return c - '0';
  if (c >= 'a' && c <= 'f') return c - 'a' + 10;
  if (c >= 'A' && c <= 'F') return c - 'A' + 10;
  return -1;
}

// Reads the grammar file format: line directives "start NAME" and
// "token NAME /regex/|"literal" [ignore] [category] [nocase] [prio N]", and
// free-form rules "lhs : a b @label | %empty ;".  '#' starts a comment.
static GrammarFile read_grammar(const string& text) {
  GrammarFile gf;
  string rules_text;
  size_t pos = 0;
  int lineno = 0;
  while (pos <= text.size()) {
    size_t e = text.find('\n', pos);
    if (e == string::npos) e = text.size();
    string line = text.substr(pos, e - pos);
    pos = e + 1;
    ++lineno;
    size_t a = 0;
    while (a < line.size() && (line[a] == ' ' || line[a] == '\t' || line[a] == '\r')) ++a;
    auto word_at = [&](size_t p, const char* w) {
      size_t n = strlen(w);
      return line.compare(p, n, w) == 0 && p + n < line.size() &&
             (line[p + n] == ' ' || line[p + n] == '\t');
    };
    if (word_at(a, "start")) {
      size_t p = a + 5;
      while (p < line.size() && (line[p] == ' ' || line[p] == '\t')) ++p;
      size_t q = p;
      while (q < line.size() && is_ident_char(line[q])) ++q;
      gf.start = line.substr(p, q - p);
      continue;
    }
    if (word_at(a, "token")) {
      TermDecl td;
      size_t p = a + 5;
      while (p < line.size() && (line[p] == ' ' || line[p] == '\t')) ++p;
      size_t q = p;
      while (q < line.size() && is_ident_char(line[q])) ++q;
      td.name = line.substr(p, q - p);
      if (td.name.empty()) throw OracleError("line " + std::to_string(lineno) + ": token name");
      p = q;
      while (p < line.size() && (line[p] == ' ' || line[p] == '\t')) ++p;
      if (p >= line.size()) throw OracleError("line " + std::to_string(lineno) + ": pattern");
      if (line[p] == '/') {
        td.is_regex = true;
        ++p;
        string src;
        while (p < line.size() && line[p] != '/') {
          if (line[p] == '\\' && p + 1 < line.size()) {
            src += line[p];
            src += line[p + 1];
            p += 2;
          } else {
            src += line[p++];
          }
        }
        if (p >= line.size()) throw OracleError("line " + std::to_string(lineno) + ": unterminated regex");
        ++p;
        td.pattern = src;
        td.prio = 0;
      } else if (line[p] == '"') {
        ++p;
        string lit;
        while (p < line.size() && line[p] != '"') {
          if (line[p] == '\\' && p + 1 < line.size()) {
            char c = line[p + 1];
            if (c == 'n') lit += '\n';
            else if (c == 't') lit += '\t';
            else if (c == 'r') lit += '\r';
            else if (c == 'x' && p + 3 < line.size()) {
              lit += (char)(hexval(line[p + 2]) * 16 + hexval(line[p + 3]));
              p += 2;
            } else lit += c;
            p += 2;
          } else {
            lit += line[p++];
          }
        }
        if (p >= line.size()) throw OracleError("line " + std::to_string(lineno) + ": unterminated literal");
        ++p;
        td.pattern = lit;
        td.prio = 1;
      } else {
        throw OracleError("line " + std::to_string(lineno) + ": bad pattern");
      }
      // options
      while (true) {
        while (p < line.size() && (line[p] == ' ' || line[p] == '\t' || line[p] == '\r')) ++p;
        if (p >= line.size() || line[p] == '#') break;
        size_t q2 = p;
        while (q2 < line.size() && !(line[q2] == ' ' || line[q2] == '\t' || line[q2] == '\r')) ++q2;
        string opt = line.substr(p, q2 - p);
        p = q2;
        if (opt == "ignore") td.ignore = true;
        else if (opt == "category") td.category = true;
        else if (opt == "nocase") td.nocase = true;
        else if (opt == "prio") {
          while (p < line.size() && line[p] == ' ') ++p;
          size_t q3 = p;
          while (q3 < line.size() && (isdigit((unsigned char)line[q3]) || line[q3] == '-')) ++q3;
          td.prio = std::stoi(line.substr(p, q3 - p));
          p = q3;
        } else {
          throw OracleError("line " + std::to_string(lineno) + ": unknown option " + opt);
        }
      }
      gf.terms.push_back(td);
      continue;
    }
    size_t h = line.find('#');
    rules_text += (h == string::npos ? line : line.substr(0, h));
    rules_text += '\n';
  }
  if (gf.start.empty()) throw OracleError("no start symbol");
  std::map<string, int> term_id;
  for (size_t i = 0; i < gf.terms.size(); ++i) {
    if (term_id.count(gf.terms[i].name)) throw OracleError("duplicate token " + gf.terms[i].name);
    term_id[gf.terms[i].name] = (int)i;
  }
  // rules: tokens
  vector<string> toks;
  for (size_t p = 0; p < rules_text.size();) {
    char c = rules_text[p];
    if (c == ' ' || c == '\t' || c == '\n' || c == '\r') { ++p; continue; }
    if (c == ':' || c == '|' || c == ';') { toks.push_back(string(1, c)); ++p; continue; }
    if (c == '@' || c == '%' || is_ident_char(c)) {
      size_t q = p + 1;
      while (q < rules_text.size() && is_ident_char(rules_text[q])) ++q;
      toks.push_back(rules_text.substr(p, q - p));
      p = q;
      continue;
    }
    throw OracleError(string("unexpected character in rules: ") + c);
  }
  std::map<string, int> nt_id;
  // first pass: every rule lhs is a nonterminal
  for (size_t i = 0; i + 1 < toks.size(); ++i)
    if (toks[i + 1] == ":" && !nt_id.count(toks[i])) {
      if (term_id.count(toks[i])) throw OracleError("rule for a token: " + toks[i]);
      nt_id[toks[i]] = (int)gf.nonterms.size();
      gf.nonterms.push_back(toks[i]);
    }
  const int T = (int)gf.terms.size();
  size_t i = 0;
  while (i < toks.size()) {
    if (i + 1 >= toks.size() || toks[i + 1] != ":") throw OracleError("expected 'name :' near " + toks[i]);
    int lhs = nt_id[toks[i]];
    i += 2;
    Rule cur{lhs, {}, ""};
    bool empty_mark = false;
    while (true) {
      if (i >= toks.size()) throw OracleError("unterminated rule");
      const string& t = toks[i];
      if (t == "|" || t == ";") {
        if (empty_mark && !cur.rhs.empty()) throw OracleError("%empty with symbols");
        gf.rules.push_back(cur);
        cur = Rule{lhs, {}, ""};
        empty_mark = false;
        ++i;
        if (t == ";") break;
        continue;
      }
      if (t == "%empty") { empty_mark = true; ++i; continue; }
      if (t[0] == '@') { cur.label = t.substr(1); ++i; continue; }
      auto ti = term_id.find(t);
      if (ti != term_id.end()) cur.rhs.push_back(ti->second);
      else {
        auto ni = nt_id.find(t);
        if (ni == nt_id.end()) throw OracleError("undefined symbol " + t);
        cur.rhs.push_back(T + ni->second);
      }
      ++i;
    }
  }
  if (!nt_id.count(gf.start)) throw OracleError("start symbol has no rules");
  return gf;
}

// --------------------------------------------------------------- Thompson NFA
struct NState {
  std::bitset<256> on;   // byte set of the single labelled edge (if next >= 0)
  int next = -1;
  vector<int> eps;
  int accept = -1;       // terminal id accepted here
};

struct Nfa {
  vector<NState> st;
  int start = -1;
  int add() { st.emplace_back(); return (int)st.size() - 1; }
};

struct Frag { int in, out; };

// Regex syntax: literal bytes, \n \t \r \xHH and backslash-escaped
// punctuation, '.', classes [..] / [^..] with ranges, grouping, |, *, +, ?.
struct RegexReader {
  const string& s;
  size_t p = 0;
  Nfa& nfa;
  RegexReader(const string& src, Nfa& n) : s(src), nfa(n) {}

  int escaped(size_t& q) {
    char c = s[q + 1];
    q += 2;
    if (c == 'n') return '\n';
    if (c == 't') return '\t';
    if (c == 'r') return '\r';
    if (c == 'x') {
      if (q + 1 >= s.size()) throw OracleError("bad \\x escape");
      int v = hexval(s[q]) * 16 + hexval(s[q + 1]);
      q += 2;
      return v;
    }
    return (unsigned char)c;
  }
  Frag edge(const std::bitset<256>& on) {
    int a = nfa.add(), b = nfa.add();
    nfa.st[a].on = on;
    nfa.st[a].next = b;
    return {a, b};
  }
  Frag alt() {
    Frag f = concat();
    while (p < s.size() && s[p] == '|') {
      ++p;
      Frag g = concat();
      int a = nfa.add(), b = nfa.add();
      nfa.st[a].eps = {f.in, g.in};
      nfa.st[f.out].eps.push_back(b);
      nfa.st[g.out].eps.push_back(b);
      f = {a, b};
    }
    return f;
  }
  Frag concat() {
    int a = nfa.add();
    Frag f{a, a};
    while (p < s.size() && s[p] != '|' && s[p] != ')') {
      Frag g = repeat();
      nfa.st[f.out].eps.push_back(g.in);
      f.out = g.out;
    }
    return f;
  }
  Frag repeat() {
    Frag f = atom();
    while (p < s.size() && (s[p] == '*' || s[p] == '+' || s[p] == '?')) {
      char op = s[p++];
      int a = nfa.add(), b = nfa.add();
      nfa.st[a].eps.push_back(f.in);
      nfa.st[f.out].eps.push_back(b);
      if (op == '*' || op == '?') nfa.st[a].eps.push_back(b);
      if (op == '*' || op == '+') nfa.st[f.out].eps.push_back(f.in);
      f = {a, b};
    }
    return f;
  }
  Frag atom() {
    if (p >= s.size()) throw OracleError("regex ends early");
    char c = s[p];
    if (c == '(') {
      ++p;
      Frag f = alt();
      if (p >= s.size() || s[p] != ')') throw OracleError("missing )");
      ++p;
      return f;
    }
    std::bitset<256> on;
    if (c == '.') {
      ++p;
      on.set();
      return edge(on);
    }
    if (c == '[') {
      ++p;
      bool neg = false;
      if (p < s.size() && s[p] == '^') { neg = true; ++p; }
      bool first = true;
      while (p < s.size() && (s[p] != ']' || first)) {
        first = false;
        int lo;
        if (s[p] == '\\') lo = escaped(p);
        else lo = (unsigned char)s[p++];
        int hi = lo;
        if (p + 1 < s.size() && s[p] == '-' && s[p + 1] != ']') {
          ++p;
          if (s[p] == '\\') hi = escaped(p);
          else hi = (unsigned char)s[p++];
        }
        if (hi < lo) throw OracleError("bad class range");
        for (int b = lo; b <= hi; ++b) on.set(b);
      }
      if (p >= s.size()) throw OracleError("unterminated class");
      ++p;
      if (neg) on.flip();
      return edge(on);
    }
    if (c == '*' || c == '+' || c == '?' || c == ')' || c == '|') throw OracleError("misplaced operator");
    int b;
    if (c == '\\') b = escaped(p);
    else b = (unsigned char)s[p++];
    on.set(b);
    return edge(on);
  }
};

static Frag literal_frag(Nfa& nfa, const string& lit, bool nocase) {
  int a = nfa.add();
  Frag f{a, a};
  for (unsigned char c : lit) {
    std::bitset<256> on;
    on.set(c);
    if (nocase && c >= 'a' && c <= 'z') on.set(c - 32);
    if (nocase && c >= 'A' && c <= 'Z') on.set(c + 32);
    int x = nfa.add(), y = nfa.add();
    nfa.st[x].on = on;
    nfa.st[x].next = y;
    nfa.st[f.out].eps.push_back(x);
    f.out = y;
  }
  return f;
}

// ------------------------------------------------------------------ grammar+
struct Grammar {
  GrammarFile gf;
  int T = 0;                       // terminal count
  int NT = 0;                      // nonterminal count
  vector<Rule> rules;              // after projection and reduction
  vector<vector<int>> rules_of;    // nonterminal -> rule indices
  vector<char> nullable;           // per nonterminal
  int start_nt = -1;
  Nfa nfa;
  vector<vector<int>> reach_terms; // NFA state -> terminals whose accept is reachable
  vector<int> prio;
  vector<char> ignored, category;

  // per-call scratch for single-threaded entry points
  std::mutex mu;
};

static void build_grammar(Grammar& G, const string& text, const string& drops_csv) {
  G.gf = read_grammar(text);
  G.T = (int)G.gf.terms.size();
  G.NT = (int)G.gf.nonterms.size();
  std::set<string> drops;
  {
    string cur;
    for (char c : drops_csv + ",") {
      if (c == ',') { if (!cur.empty()) drops.insert(cur); cur.clear(); }
      else if (c != ' ') cur += c;
    }
  }
  vector<Rule> kept;
  for (auto& r : G.gf.rules)
    if (r.label.empty() || !drops.count(r.label)) kept.push_back(r);
  for (auto& d : drops) {
    bool found = false;
    for (auto& r : G.gf.rules) if (r.label == d) found = true;
    if (!found) throw OracleError("projection names unknown label " + d);
  }
  // useless-symbol elimination: generating, then reachable
  vector<char> gen(G.NT, 0);
  for (bool ch = true; ch;) {
    ch = false;
    for (auto& r : kept) {
      if (gen[r.lhs]) continue;
      bool ok = true;
      for (int s : r.rhs) if (s >= G.T && !gen[s - G.T]) ok = false;
      if (ok) { gen[r.lhs] = 1; ch = true; }
    }
  }
  int st = -1;
  for (int i = 0; i < G.NT; ++i) if (G.gf.nonterms[i] == G.gf.start) st = i;
  if (!gen[st]) throw OracleError("empty language after projection");
  vector<Rule> gen_rules;
  for (auto& r : kept) {
    bool ok = gen[r.lhs];
    for (int s : r.rhs) if (s >= G.T && !gen[s - G.T]) ok = false;
    if (ok) gen_rules.push_back(r);
  }
  vector<char> reach(G.NT, 0);
  reach[st] = 1;
  for (bool ch = true; ch;) {
    ch = false;
    for (auto& r : gen_rules) {
      if (!reach[r.lhs]) continue;
      for (int s : r.rhs)
        if (s >= G.T && !reach[s - G.T]) { reach[s - G.T] = 1; ch = true; }
    }
  }
  G.rules.clear();
  for (auto& r : gen_rules) if (reach[r.lhs]) G.rules.push_back(r);
  G.start_nt = st;
  G.rules_of.assign(G.NT, {});
  for (size_t i = 0; i < G.rules.size(); ++i) G.rules_of[G.rules[i].lhs].push_back((int)i);
  G.nullable.assign(G.NT, 0);
  for (bool ch = true; ch;) {
    ch = false;
    for (auto& r : G.rules) {
      if (G.nullable[r.lhs]) continue;
      bool ok = true;
      for (int s : r.rhs) if (s < G.T || !G.nullable[s - G.T]) ok = false;
      if (ok) { G.nullable[r.lhs] = 1; ch = true; }
    }
  }
  // NFA over every declared terminal
  G.nfa = Nfa();
  G.nfa.start = G.nfa.add();
  G.prio.resize(G.T);
  G.ignored.resize(G.T);
  G.category.resize(G.T);
  for (int t = 0; t < G.T; ++t) {
    const TermDecl& d = G.gf.terms[t];
    Frag f;
    if (d.is_regex) {
      if (d.nocase) throw OracleError("nocase applies to literals only");
      RegexReader rr(d.pattern, G.nfa);
      f = rr.alt();
      if (rr.p != d.pattern.size()) throw OracleError("regex trailing input in " + d.name);
    } else {
      if (d.pattern.empty()) throw OracleError("empty literal " + d.name);
      f = literal_frag(G.nfa, d.pattern, d.nocase);
    }
    G.nfa.st[f.out].accept = t;
    G.nfa.st[G.nfa.start].eps.push_back(f.in);
    G.prio[t] = d.prio;
    G.ignored[t] = d.ignore;
    G.category[t] = d.category;
  }
  // which accepts are reachable from each NFA state (plain graph search)
  const int S = (int)G.nfa.st.size();
  G.reach_terms.assign(S, {});
  for (int s = 0; s < S; ++s) {
    vector<char> seen(S, 0);
    vector<int> stack{s};
    seen[s] = 1;
    std::set<int> terms;
    while (!stack.empty()) {
      int u = stack.back();
      stack.pop_back();
      const NState& ns = G.nfa.st[u];
      if (ns.accept >= 0) terms.insert(ns.accept);
      if (ns.next >= 0 && ns.on.any() && !seen[ns.next]) { seen[ns.next] = 1; stack.push_back(ns.next); }
      for (int v : ns.eps) if (!seen[v]) { seen[v] = 1; stack.push_back(v); }
    }
    G.reach_terms[s].assign(terms.begin(), terms.end());
  }
}

// ------------------------------------------------------- NFA simulation cache
// State sets are epsilon-closed sorted vectors; step results are memoized so
// that repeated simulation is cheap.  One cache per thread.
struct LexCache {
  const Grammar* G = nullptr;
  vector<vector<int>> sets;
  std::map<vector<int>, int> ids;
  vector<vector<int>> step;        // set id -> 256 successors (-1 unknown)
  vector<vector<int>> accepts;     // set id -> terminals accepted
  vector<vector<int>> live;        // set id -> terminals with a reachable accept
  int start = -1, empty = -1;

  void init(const Grammar* g) {
    G = g;
    sets.clear(); ids.clear(); step.clear(); accepts.clear(); live.clear();
    empty = intern({});
    start = intern(closure({G->nfa.start}));
  }
  vector<int> closure(vector<int> seed) const {
    std::set<int> out(seed.begin(), seed.end());
    vector<int> stack(seed.begin(), seed.end());
    while (!stack.empty()) {
      int u = stack.back();
      stack.pop_back();
      for (int v : G->nfa.st[u].eps)
        if (out.insert(v).second) stack.push_back(v);
    }
    return vector<int>(out.begin(), out.end());
  }
  int intern(const vector<int>& s) {
    auto it = ids.find(s);
    if (it != ids.end()) return it->second;
    int id = (int)sets.size();
    ids[s] = id;
    sets.push_back(s);
    step.emplace_back(256, -1);
    std::set<int> acc, lv;
    for (int u : s) {
      if (G->nfa.st[u].accept >= 0) acc.insert(G->nfa.st[u].accept);
      for (int t : G->reach_terms[u]) lv.insert(t);
    }
    accepts.emplace_back(acc.begin(), acc.end());
    live.emplace_back(lv.begin(), lv.end());
    return id;
  }
  int next(int id, unsigned char b) {
    int r = step[id][b];
    if (r >= 0) return r;
    vector<int> moved;
    for (int u : sets[id]) {
      const NState& ns = G->nfa.st[u];
      if (ns.next >= 0 && ns.on.test(b)) moved.push_back(ns.next);
    }
    r = intern(closure(moved));
    step[id][b] = r;
    return r;
  }
};

// ------------------------------------------------------------------ lexicon
struct Lexicon {
  // terminal id -> allow-list (absent: unrestricted)
  std::map<int, std::unordered_set<string>> words;
  std::map<int, vector<string>> sorted;
  bool restricts(int t) const { return words.count(t) != 0; }
  bool is_word(int t, const string& s) const { return words.at(t).count(s) != 0; }
  bool is_prefix(int t, const string& s) const {
    const vector<string>& v = sorted.at(t);
    auto it = std::lower_bound(v.begin(), v.end(), s);
    return it != v.end() && it->compare(0, s.size(), s) == 0;
  }
};

// -------------------------------------------------------------------- Earley
struct Item {
  int rule, dot, origin;
};

struct ESet {
  vector<Item> items;
  std::unordered_set<uint64_t> seen;
  bool add(const Item& it) {
    uint64_t k = ((uint64_t)it.rule << 40) | ((uint64_t)it.dot << 32) | (uint32_t)it.origin;
    if (!seen.insert(k).second) return false;
    items.push_back(it);
    return true;
  }
};

// A chart whose first sets may be a shared read-only base (checkpoint mode).
struct Chart {
  const vector<ESet>* base = nullptr;
  vector<ESet> own;
  size_t size() const { return (base ? base->size() : 0) + own.size(); }
  const ESet& at(size_t i) const {
    size_t nb = base ? base->size() : 0;
    return i < nb ? (*base)[i] : own[i - nb];
  }
  ESet& last_own() { return own.back(); }
};

struct Parser {
  const Grammar& G;
  explicit Parser(const Grammar& g) : G(g) {}

  int next_sym(const Item& it) const {
    const Rule& r = G.rules[it.rule];
    return it.dot < (int)r.rhs.size() ? r.rhs[it.dot] : -1;
  }
  // predict / complete until the set (the chart's last, owned set) is closed
  void close(Chart& ch) const {
    size_t k = ch.size() - 1;
    ESet& cur = ch.last_own();
    for (size_t i = 0; i < cur.items.size(); ++i) {
      Item it = cur.items[i];
      int x = next_sym(it);
      if (x < 0) {  // complete
        int lhs = G.rules[it.rule].lhs;
        if ((size_t)it.origin == k) {
          for (size_t j = 0; j < cur.items.size(); ++j) {
            const Item& p = cur.items[j];
            if (next_sym(p) == G.T + lhs) cur.add({p.rule, p.dot + 1, p.origin});
          }
        } else {
          const ESet& org = ch.at(it.origin);
          for (const Item& p : org.items)
            if (next_sym(p) == G.T + lhs) cur.add({p.rule, p.dot + 1, p.origin});
        }
      } else if (x >= G.T) {  // predict
        int nt = x - G.T;
        for (int r : G.rules_of[nt]) cur.add({r, 0, (int)k});
        if (G.nullable[nt]) cur.add({it.rule, it.dot + 1, it.origin});
      }
    }
  }
  void init(Chart& ch) const {
    ch.own.emplace_back();
    for (int r : G.rules_of[G.start_nt]) ch.last_own().add({r, 0, 0});
    close(ch);
  }
  // shift terminal t; false if no item expects it
  bool scan(Chart& ch, int t) const {
    const ESet& cur = ch.at(ch.size() - 1);
    ESet nxt;
    for (const Item& it : cur.items)
      if (next_sym(it) == t) nxt.add({it.rule, it.dot + 1, it.origin});
    if (nxt.items.empty()) return false;
    ch.own.push_back(std::move(nxt));
    close(ch);
    return true;
  }
  bool expects(const Chart& ch, int t) const {
    for (const Item& it : ch.at(ch.size() - 1).items)
      if (next_sym(it) == t) return true;
    return false;
  }
  bool accepted(const Chart& ch) const {
    for (const Item& it : ch.at(ch.size() - 1).items)
      if (it.origin == 0 && next_sym(it) < 0 && G.rules[it.rule].lhs == G.start_nt) return true;
    return false;
  }
};

// ---------------------------------------------------- lex + parse of a string
struct Scan {
  bool rejected = false;
  size_t rem_start = 0;   // start of the pending (trailing) lexeme
  int rem_set = -1;       // NFA set after the pending lexeme
};

struct Engine {
  const Grammar& G;
  const Lexicon* lex;
  LexCache& lc;
  Parser P;
  Engine(const Grammar& g, const Lexicon* l, LexCache& c) : G(g), lex(l), lc(c), P(g) {}

  bool lexicon_ok_word(int t, const string& s) const {
    return !(G.category[t] && lex && lex->restricts(t)) || lex->is_word(t, s);
  }
  bool lexicon_ok_prefix(int t, const string& s) const {
    return !(G.category[t] && lex && lex->restricts(t)) || lex->is_prefix(t, s);
  }
  // the winner among the terminals accepting the lexeme, or -1
  int resolve(const vector<int>& cands, const string& lexeme, const Chart& ch) const {
    int best = -1;
    for (int t : cands) {
      if (!lexicon_ok_word(t, lexeme)) continue;
      if (!(G.ignored[t] || P.expects(ch, t))) continue;
      if (best < 0 || G.prio[t] > G.prio[best] || (G.prio[t] == G.prio[best] && t < best)) best = t;
    }
    return best;
  }
  // Maximal-munch lexing of s[0..n) interleaved with parsing into ch.  With
  // at_eof the end of input acts as a killing byte for the pending lexeme.
  Scan run(const uint8_t* s, size_t n, Chart& ch, bool at_eof) const {
    Scan out;
    size_t i = 0;
    while (true) {
      int S = lc.start;
      long last_len = -1;
      int last_S = -1;
      size_t j = i;
      while (j < n) {
        int S2 = lc.next(S, s[j]);
        if (S2 == lc.empty) break;
        S = S2;
        ++j;
        if (!lc.accepts[S].empty()) { last_len = (long)(j - i); last_S = S; }
      }
      if (j == n && !(at_eof && i < n)) {
        out.rem_start = i;
        out.rem_set = S;
        return out;
      }
      if (last_len < 0) { out.rejected = true; return out; }
      string lexeme((const char*)s + i, (size_t)last_len);
      int w = resolve(lc.accepts[last_S], lexeme, ch);
      if (w < 0) { out.rejected = true; return out; }
      if (!G.ignored[w] && !P.scan(ch, w)) { out.rejected = true; return out; }
      i += (size_t)last_len;
    }
  }
  // Definition 2's trailing test on the pending lexeme s[rem_start..n).
  bool trailing_viable(const uint8_t* s, size_t n, const Scan& sc, const Chart& ch) const {
    if (sc.rejected) return false;
    if (sc.rem_start == n) return true;
    string r((const char*)s + sc.rem_start, n - sc.rem_start);
    for (int t : lc.live[sc.rem_set]) {
      if (!(G.ignored[t] || P.expects(ch, t))) continue;
      if (lexicon_ok_prefix(t, r)) return true;
    }
    return false;
  }
  bool viable(const uint8_t* s, size_t n) const {
    Chart ch;
    P.init(ch);
    Scan sc = run(s, n, ch, false);
    return trailing_viable(s, n, sc, ch);
  }
  bool member(const uint8_t* s, size_t n) const {
    Chart ch;
    P.init(ch);
    Scan sc = run(s, n, ch, true);
    return !sc.rejected && P.accepted(ch);
  }
};

struct OGrammar {
  Grammar G;
  LexCache single;
  vector<LexCache> per_thread;
};

struct OVocab {
  vector<string> spell;
  vector<char> special;
  int eos = -1;
};

void set_err(char* err, int len, const string& m) {
  if (err && len > 0) {
    strncpy(err, m.c_str(), (size_t)len - 1);
    err[len - 1] = 0;
  }
}

}  // namespace

extern "C" {

void* oracle_grammar_new(const char* text, const char* drops, char* err, int err_len) {
  try {
    std::unique_ptr<OGrammar> og(new OGrammar());  // freed when the build throws
    build_grammar(og->G, text ? text : "", drops ? drops : "");
    og->single.init(&og->G);
    return og.release();
  } catch (const std::exception& e) {
    set_err(err, err_len, e.what());
    return nullptr;
  }
}

void oracle_grammar_free(void* g) { delete (OGrammar*)g; }

int oracle_num_terminals(void* g) { return ((OGrammar*)g)->G.T; }

const char* oracle_terminal_name(void* g, int id) {
  auto* og = (OGrammar*)g;
  if (id < 0 || id >= og->G.T) return "";
  return og->G.gf.terms[id].name.c_str();
}

void* oracle_lexicon_new(void* g, int n, const char** names, const char** words, char* err,
                         int err_len) {
  auto* og = (OGrammar*)g;
  auto* lx = new Lexicon();
  for (int i = 0; i < n; ++i) {
    int t = -1;
    for (int k = 0; k < og->G.T; ++k) if (og->G.gf.terms[k].name == names[i]) t = k;
    if (t < 0 || !og->G.category[t]) {
      set_err(err, err_len, string("not a category terminal: ") + names[i]);
      delete lx;
      return nullptr;
    }
    auto& set = lx->words[t];
    string cur;
    for (const char* p = words[i];; ++p) {
      if (*p == '\n' || *p == 0) {
        if (!cur.empty()) set.insert(cur);
        cur.clear();
        if (*p == 0) break;
      } else {
        cur += *p;
      }
    }
    lx->sorted[t] = vector<string>(set.begin(), set.end());
    std::sort(lx->sorted[t].begin(), lx->sorted[t].end());
  }
  return lx;
}

void oracle_lexicon_free(void* lex) { delete (Lexicon*)lex; }

void* oracle_vocab_new(const uint8_t* bytes, const uint64_t* offsets, int V,
                       const int32_t* special_ids, int n_special, int32_t eos_id) {
  auto* v = new OVocab();
  v->spell.resize(V);
  v->special.assign(V, 0);
  for (int i = 0; i < V; ++i)
    v->spell[i].assign((const char*)bytes + offsets[i], (size_t)(offsets[i + 1] - offsets[i]));
  for (int i = 0; i < n_special; ++i)
    if (special_ids[i] >= 0 && special_ids[i] < V) v->special[special_ids[i]] = 1;
  v->eos = eos_id;
  if (eos_id >= 0 && eos_id < V) v->special[eos_id] = 1;
  return v;
}

void oracle_vocab_free(void* voc) { delete (OVocab*)voc; }

int oracle_mask(void* g, void* lexp, void* vocp, const uint8_t* w, size_t n, int mode,
                const int32_t* token_ids, int n_tokens, uint32_t* out_words, uint8_t* out_bits,
                int32_t* eos_ok, int nthreads) {
  auto* og = (OGrammar*)g;
  const Grammar& G = og->G;
  const Lexicon* lex = (const Lexicon*)lexp;
  const OVocab& voc = *(const OVocab*)vocp;
  const int V = (int)voc.spell.size();
  const bool all = token_ids == nullptr;
  const int count = all ? V : n_tokens;
#ifdef _OPENMP
  int nt = nthreads > 0 ? nthreads : omp_get_max_threads();
#else
  int nt = 1;
  (void)nthreads;
#endif
  if ((int)og->per_thread.size() < nt) {
    og->per_thread.resize(nt);
    for (auto& c : og->per_thread) if (!c.G) c.init(&G);
  }
  vector<uint8_t> bits(count, 0);

  // end of sequence: w in L
  {
    Engine e(G, lex, og->single);
    *eos_ok = e.member(w, n) ? 1 : 0;
  }
  // checkpoint: the chart after w's completed lexemes, and the pending lexeme
  Chart base_chart;
  Scan base_scan;
  if (mode == 1) {
    Engine e(G, lex, og->single);
    e.P.init(base_chart);
    base_scan = e.run(w, n, base_chart, false);
  }
  vector<ESet> base_sets;
  if (mode == 1) base_sets = std::move(base_chart.own);
  const string rem = mode == 1 && !base_scan.rejected
                         ? string((const char*)w + base_scan.rem_start, n - base_scan.rem_start)
                         : string();

#pragma omp parallel for schedule(dynamic, 64) num_threads(nt)
  for (int i = 0; i < count; ++i) {
    int tid = 0;
#ifdef _OPENMP
    tid = omp_get_thread_num();
#endif
    int t = all ? i : token_ids[i];
    if (t < 0 || t >= V || voc.special[t] || voc.spell[t].empty()) continue;
    Engine e(G, lex, og->per_thread[tid]);
    const string& sp = voc.spell[t];
    if (mode == 0) {
      string s((const char*)w, n);
      s += sp;
      bits[i] = e.viable((const uint8_t*)s.data(), s.size()) ? 1 : 0;
    } else {
      if (base_scan.rejected) continue;
      string s = rem + sp;
      Chart ch;
      ch.base = &base_sets;
      Scan sc = e.run((const uint8_t*)s.data(), s.size(), ch, false);
      bits[i] = e.trailing_viable((const uint8_t*)s.data(), s.size(), sc, ch) ? 1 : 0;
    }
  }
  if (all) {
    const int W = (V + 31) / 32;
    for (int k = 0; k < W; ++k) out_words[k] = 0;
    for (int t = 0; t < V; ++t)
      if (bits[t]) out_words[t >> 5] |= 1u << (t & 31);
    if (voc.eos >= 0 && voc.eos < V && *eos_ok) out_words[voc.eos >> 5] |= 1u << (voc.eos & 31);
  } else {
    for (int i = 0; i < count; ++i) {
      int t = token_ids[i];
      out_bits[i] = (t == voc.eos && t >= 0) ? (uint8_t)*eos_ok : bits[i];
    }
  }
  return 0;
}

int oracle_viable(void* g, void* lex, const uint8_t* w, size_t n) {
  auto* og = (OGrammar*)g;
  Engine e(og->G, (const Lexicon*)lex, og->single);
  return e.viable(w, n) ? 1 : 0;
}

int oracle_member(void* g, void* lex, const uint8_t* w, size_t n) {
  auto* og = (OGrammar*)g;
  Engine e(og->G, (const Lexicon*)lex, og->single);
  return e.member(w, n) ? 1 : 0;
}

int oracle_allowed(void* g, void* lex, const uint8_t* w, size_t n, uint8_t* out) {
  auto* og = (OGrammar*)g;
  Engine e(og->G, (const Lexicon*)lex, og->single);
  Chart ch;
  e.P.init(ch);
  Scan sc = e.run(w, n, ch, false);
  for (int t = 0; t < og->G.T; ++t) out[t] = (!sc.rejected && e.P.expects(ch, t)) ? 1 : 0;
  return sc.rejected ? 0 : 1;
}

}  // extern "C"
