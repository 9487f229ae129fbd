// grammar.cpp -- reads the grammar text format.
//
// Format (line directives, free-form rules):
//   start NAME
//   token NAME /regex/   [ignore] [category] [prio N]
//   token NAME "literal" [ignore] [category] [nocase] [prio N]
//   lhs : sym sym @label | %empty ;
// '#' begins a comment.  Literal tokens default to priority 1, regex tokens to
// 0 (the contextual-resolution order of section 2, L1).  Terminal ids follow
// declaration order and are never renumbered (section 4.3, T2 tier).
#include <cctype>
#include <cstring>

#include "host.h"

namespace grid {
namespace {

struct Cursor {
  const std::string& s;
  size_t i = 0;
  int line = 1;
  explicit Cursor(const std::string& t) : s(t) {}
  bool eof() const { return i >= s.size(); }
  char peek() const { return i < s.size() ? s[i] : '\0'; }
  [[noreturn]] void fail(const std::string& m) const {
    throw Error(GRID_E_GRAMMAR_SYNTAX, "grammar line " + std::to_string(line) + ": " + m);
  }
  void skip_blanks() {  // spaces and tabs only
    while (!eof() && (s[i] == ' ' || s[i] == '\t' || s[i] == '\r')) ++i;
  }
  void skip_comment() {
    if (peek() == '#')
      while (!eof() && s[i] != '\n') ++i;
  }
  bool at_eol() {
    skip_blanks();
    skip_comment();
    return eof() || s[i] == '\n';
  }
  std::string word() {
    size_t b = i;
    while (!eof() && (isalnum((unsigned char)s[i]) || s[i] == '_')) ++i;
    return s.substr(b, i - b);
  }
};

int hex_digit(char c) {
  if (c >= '0' && c <= '9') return c - '0';
  c = (char)tolower((unsigned char)c);
  if (c >= 'a' && c <= 'f') return c - 'a' + 10;
  return -1;
}

void read_token_decl(Cursor& c, GrammarText& g) {
  Terminal t;
  c.skip_blanks();
  t.name = c.word();
  if (t.name.empty()) c.fail("token needs a name");
  c.skip_blanks();
  char open = c.peek();
  if (open == '/') {
    t.regex = true;
    ++c.i;
    while (!c.eof() && c.peek() != '/' && c.peek() != '\n') {
      if (c.peek() == '\\') {
        if (c.i + 1 >= c.s.size()) c.fail("dangling escape");
        t.source.push_back(c.s[c.i]);
        t.source.push_back(c.s[c.i + 1]);
        c.i += 2;
      } else {
        t.source.push_back(c.s[c.i++]);
      }
    }
    if (c.peek() != '/') c.fail("unterminated regex");
    ++c.i;
    t.priority = 0;
  } else if (open == '"') {
    ++c.i;
    while (!c.eof() && c.peek() != '"' && c.peek() != '\n') {
      char ch = c.s[c.i++];
      if (ch != '\\') {
        t.source.push_back(ch);
        continue;
      }
      char e = c.peek();
      ++c.i;
      switch (e) {
        case 'n': t.source.push_back('\n'); break;
        case 't': t.source.push_back('\t'); break;
        case 'r': t.source.push_back('\r'); break;
        case 'x': {
          int h = hex_digit(c.peek()), l = c.i + 1 < c.s.size() ? hex_digit(c.s[c.i + 1]) : -1;
          if (h < 0 || l < 0) c.fail("bad \\x escape");
          t.source.push_back((char)(h * 16 + l));
          c.i += 2;
          break;
        }
        default: t.source.push_back(e);
      }
    }
    if (c.peek() != '"') c.fail("unterminated literal");
    ++c.i;
    if (t.source.empty()) c.fail("empty literal");
    t.priority = 1;
  } else {
    c.fail("token pattern must be /regex/ or \"literal\"");
  }
  while (!c.at_eol()) {
    std::string opt = c.word();
    if (opt == "ignore") t.ignored = true;
    else if (opt == "category") t.category = true;
    else if (opt == "nocase") t.nocase = true;
    else if (opt == "prio") {
      c.skip_blanks();
      bool neg = false;
      if (c.peek() == '-') { neg = true; ++c.i; }
      std::string num = c.word();
      if (num.empty() || !isdigit((unsigned char)num[0])) c.fail("prio needs a number");
      t.priority = (neg ? -1 : 1) * std::stoi(num);
    } else {
      c.fail("unknown token option '" + opt + "'");
    }
  }
  if (t.nocase && t.regex) c.fail("nocase applies to literal tokens only");
  for (auto& o : g.terminals)
    if (o.name == t.name) c.fail("token declared twice: " + t.name);
  g.terminals.push_back(t);
}

}  // namespace

GrammarText parse_grammar(const std::string& text) {
  GrammarText g;
  Cursor c(text);
  std::string start_name;
  // Rule text is collected as (line, token) pairs and parsed afterwards, once
  // every terminal is known.
  std::vector<std::pair<int, std::string>> rule_toks;
  while (!c.eof()) {
    c.skip_blanks();
    if (c.peek() == '#') { c.skip_comment(); continue; }
    if (c.peek() == '\n') { ++c.i; ++c.line; continue; }
    if (c.eof()) break;
    size_t save = c.i;
    std::string w = c.word();
    bool directive = (w == "token" || w == "start") && (c.peek() == ' ' || c.peek() == '\t');
    if (directive && w == "token") {
      read_token_decl(c, g);
      continue;
    }
    if (directive && w == "start") {
      c.skip_blanks();
      start_name = c.word();
      if (start_name.empty() || !c.at_eol()) c.fail("start needs one name");
      continue;
    }
    c.i = save;
    // rule material up to the end of this line
    while (!c.at_eol()) {
      char ch = c.peek();
      if (ch == ':' || ch == '|' || ch == ';') {
        rule_toks.push_back({c.line, std::string(1, ch)});
        ++c.i;
      } else if (ch == '@' || ch == '%') {
        ++c.i;
        std::string nm = c.word();
        if (nm.empty()) c.fail(std::string("'") + ch + "' needs a name");
        rule_toks.push_back({c.line, std::string(1, ch) + nm});
      } else if (isalnum((unsigned char)ch) || ch == '_') {
        rule_toks.push_back({c.line, c.word()});
      } else {
        c.fail(std::string("unexpected character '") + ch + "'");
      }
    }
  }
  if (start_name.empty()) throw Error(GRID_E_GRAMMAR_SYNTAX, "grammar has no start directive");
  if (g.terminals.empty()) throw Error(GRID_E_GRAMMAR_SYNTAX, "grammar declares no tokens");
  if ((int)g.terminals.size() > kMaxTerminals)
    throw Error(GRID_E_CAPACITY, "more than 255 terminals");

  std::map<std::string, int> term_of, nt_of;
  for (size_t k = 0; k < g.terminals.size(); ++k) term_of[g.terminals[k].name] = (int)k;
  for (size_t k = 0; k + 1 < rule_toks.size(); ++k)
    if (rule_toks[k + 1].second == ":" && !nt_of.count(rule_toks[k].second)) {
      const std::string& nm = rule_toks[k].second;
      if (term_of.count(nm))
        throw Error(GRID_E_GRAMMAR_SYNTAX, "token used as a rule head: " + nm);
      nt_of[nm] = (int)g.nonterminals.size();
      g.nonterminals.push_back(nm);
    }
  size_t k = 0;
  auto fail_at = [&](size_t at, const std::string& m) {
    int ln = at < rule_toks.size() ? rule_toks[at].first : -1;
    throw Error(GRID_E_GRAMMAR_SYNTAX, "grammar line " + std::to_string(ln) + ": " + m);
  };
  while (k < rule_toks.size()) {
    if (k + 1 >= rule_toks.size() || rule_toks[k + 1].second != ":")
      fail_at(k, "expected 'name :' before '" + rule_toks[k].second + "'");
    int lhs = nt_of[rule_toks[k].second];
    k += 2;
    Production p;
    p.lhs = lhs;
    bool empty = false;
    for (;;) {
      if (k >= rule_toks.size()) fail_at(k - 1, "rule not terminated by ';'");
      const std::string& t = rule_toks[k].second;
      ++k;
      if (t == "|" || t == ";") {
        if (empty && !p.rhs.empty()) fail_at(k - 1, "%empty alternative with symbols");
        if (!empty && p.rhs.empty()) fail_at(k - 1, "empty alternative needs %empty");
        g.productions.push_back(p);
        p = Production();
        p.lhs = lhs;
        empty = false;
        if (t == ";") break;
      } else if (t == "%empty") {
        empty = true;
      } else if (t[0] == '%') {
        fail_at(k - 1, "unknown directive " + t);
      } else if (t[0] == '@') {
        p.label = t.substr(1);
      } else if (t == ":") {
        fail_at(k - 1, "missing ';' before a new rule");
      } else if (term_of.count(t)) {
        p.rhs.push_back(term_of[t]);
      } else if (nt_of.count(t)) {
        p.rhs.push_back(~nt_of[t]);
      } else {
        fail_at(k - 1, "undefined symbol " + t);
      }
    }
  }
  if (!nt_of.count(start_name))
    throw Error(GRID_E_GRAMMAR_SYNTAX, "start symbol " + start_name + " has no rules");
  g.start = nt_of[start_name];
  return g;
}

}  // namespace grid
