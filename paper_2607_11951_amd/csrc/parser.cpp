// parser.cpp -- role projection, useless-symbol removal and LALR(1) tables.
//
// Section 2 (L2): a role keeps a subset of the productions; useless symbols
// are then removed (reducedness is what makes "the parser accepts the next
// terminal" equal "the prefix stays viable", Proposition 3) and the language
// must stay nonempty.  The LALR(1) automaton is built from the LR(0) item sets
// with lookaheads found by spontaneous generation and propagation (the
// classic kernel-item method); any shift/reduce or reduce/reduce conflict is
// an error.  Tables keep full reduce rows (no default reductions); the mask
// path computes allowed terminals by simulating reduce chains anyway
// (section 3.2), so it is exact with or without table compression.
#include <algorithm>
#include <cstring>
#include <map>
#include <set>

#include "host.h"
#include "lexhash.h"

namespace grid {
namespace {

struct Bits {  // terminal set over T+2 symbols (T = end of input, T+1 = probe)
  uint64_t w[5] = {0, 0, 0, 0, 0};
  void set(int i) { w[i >> 6] |= 1ull << (i & 63); }
  bool test(int i) const { return (w[i >> 6] >> (i & 63)) & 1; }
  bool merge(const Bits& o) {
    bool ch = false;
    for (int k = 0; k < 5; ++k) {
      uint64_t n = w[k] | o.w[k];
      ch |= n != w[k];
      w[k] = n;
    }
    return ch;
  }
};

struct G2 {  // reduced grammar with augmented production 0: S' -> S
  int T = 0, N = 0;  // N includes S' as the last nonterminal
  std::vector<int> lhs;
  std::vector<std::vector<int>> rhs;  // symbols: t < T terminal, T + n nonterminal
  std::vector<std::vector<int>> prods_of;
  std::vector<char> nullable;
  std::vector<Bits> first;
  bool is_nt(int x) const { return x >= T; }
};

using Item = uint32_t;  // prod << 8 | dot
inline Item mk(int p, int d) { return (Item)p << 8 | (Item)d; }
inline int ip(Item x) { return (int)(x >> 8); }
inline int id(Item x) { return (int)(x & 255); }

}  // namespace

void compact_tables(Parser& P);

Parser build_parser(const GrammarText& g, const std::vector<std::string>& drop) {
  const int T = (int)g.terminals.size();
  const int N0 = (int)g.nonterminals.size();
  // projection
  std::set<std::string> dropset(drop.begin(), drop.end());
  for (const auto& lab : dropset) {
    bool found = false;
    for (const auto& p : g.productions) found |= p.label == lab;
    if (!found) throw Error(GRID_E_ARG, "role projection names unknown label '" + lab + "'");
  }
  std::vector<const Production*> kept;
  for (const auto& p : g.productions)
    if (p.label.empty() || !dropset.count(p.label)) kept.push_back(&p);
  // generating nonterminals
  std::vector<char> gen(N0, 0);
  for (bool ch = true; ch;) {
    ch = false;
    for (const Production* p : kept) {
      if (gen[p->lhs]) continue;
      bool all = true;
      for (int s : p->rhs)
        if (s < 0 && !gen[~s]) { all = false; break; }
      if (all) gen[p->lhs] = ch = true;
    }
  }
  if (!gen[g.start]) throw Error(GRID_E_EMPTY_LANGUAGE, "the role projection leaves an empty language");
  std::vector<const Production*> genp;
  for (const Production* p : kept) {
    bool ok = gen[p->lhs];
    for (int s : p->rhs) ok = ok && (s >= 0 || gen[~s]);
    if (ok) genp.push_back(p);
  }
  // reachable from the start symbol
  std::vector<char> reach(N0, 0);
  reach[g.start] = 1;
  for (bool ch = true; ch;) {
    ch = false;
    for (const Production* p : genp)
      if (reach[p->lhs])
        for (int s : p->rhs)
          if (s < 0 && !reach[~s]) reach[~s] = ch = true;
  }
  std::vector<int> nt_new(N0, -1);
  int N = 0;
  for (int a = 0; a < N0; ++a)
    if (reach[a] && gen[a]) nt_new[a] = N++;

  G2 G;
  G.T = T;
  G.N = N + 1;  // + S'
  const int SP = N;
  G.lhs.push_back(SP);
  G.rhs.push_back({T + nt_new[g.start]});
  Parser out;
  out.term_used.assign(T, 0);
  for (const Production* p : genp) {
    if (!reach[p->lhs]) continue;
    G.lhs.push_back(nt_new[p->lhs]);
    std::vector<int> r;
    for (int s : p->rhs) {
      if (s >= 0) {
        r.push_back(s);
        out.term_used[s] = 1;
      } else {
        r.push_back(T + nt_new[~s]);
      }
    }
    if (r.size() > 200) throw Error(GRID_E_CAPACITY, "production longer than 200 symbols");
    G.rhs.push_back(r);
  }
  const int P = (int)G.lhs.size();
  G.prods_of.assign(G.N, {});
  for (int p = 0; p < P; ++p) G.prods_of[G.lhs[p]].push_back(p);
  // nullable and FIRST
  G.nullable.assign(G.N, 0);
  G.first.assign(G.N, Bits());
  for (bool ch = true; ch;) {
    ch = false;
    for (int p = 0; p < P; ++p) {
      int A = G.lhs[p];
      bool all_null = true;
      for (int x : G.rhs[p]) {
        if (!G.is_nt(x)) {
          Bits b;
          b.set(x);
          ch |= G.first[A].merge(b);
          all_null = false;
          break;
        }
        ch |= G.first[A].merge(G.first[x - T]);
        if (!G.nullable[x - T]) { all_null = false; break; }
      }
      if (all_null && !G.nullable[A]) G.nullable[A] = ch = true;
    }
  }
  auto first_of_seq = [&](int p, int from, const Bits& tail, Bits& out_bits) {
    for (size_t k = (size_t)from; k < G.rhs[p].size(); ++k) {
      int x = G.rhs[p][k];
      if (!G.is_nt(x)) { out_bits.set(x); return; }
      out_bits.merge(G.first[x - T]);
      if (!G.nullable[x - T]) return;
    }
    out_bits.merge(tail);
  };

  // LR(0) item sets
  auto closure0 = [&](std::vector<Item> items) {
    std::set<Item> seen(items.begin(), items.end());
    for (size_t k = 0; k < items.size(); ++k) {
      int p = ip(items[k]), d = id(items[k]);
      if (d < (int)G.rhs[p].size() && G.is_nt(G.rhs[p][d]))
        for (int q : G.prods_of[G.rhs[p][d] - T])
          if (seen.insert(mk(q, 0)).second) items.push_back(mk(q, 0));
    }
    std::sort(items.begin(), items.end());
    return items;
  };
  std::vector<std::vector<Item>> kernels;
  std::map<std::vector<Item>, int> kid;
  std::vector<std::map<int, int>> edges;  // state -> symbol -> state
  kernels.push_back({mk(0, 0)});
  kid[kernels[0]] = 0;
  for (size_t s = 0; s < kernels.size(); ++s) {
    std::vector<Item> cl = closure0(kernels[s]);
    std::map<int, std::vector<Item>> moves;
    for (Item it : cl) {
      int p = ip(it), d = id(it);
      if (d < (int)G.rhs[p].size()) moves[G.rhs[p][d]].push_back(mk(p, d + 1));
    }
    std::map<int, int> e;
    for (auto& mv : moves) {
      std::vector<Item> k = mv.second;
      std::sort(k.begin(), k.end());
      k.erase(std::unique(k.begin(), k.end()), k.end());
      auto it = kid.find(k);
      int t;
      if (it == kid.end()) {
        t = (int)kernels.size();
        kid.emplace(k, t);
        kernels.push_back(k);
      } else {
        t = it->second;
      }
      e[mv.first] = t;
    }
    edges.push_back(e);
  }
  const int NS = (int)kernels.size();
  if (NS >= 0x4000) throw Error(GRID_E_CAPACITY, "more than 16383 LR states");
  if (P >= 0x4000) throw Error(GRID_E_CAPACITY, "more than 16383 productions");

  // LR(1) closure of one item set with lookahead sets (worklist)
  const int PROBE = T + 1;
  auto closure1 = [&](const std::vector<std::pair<Item, Bits>>& seed) {
    std::map<Item, Bits> la;
    std::vector<Item> work;
    for (auto& pr : seed) {
      if (la[pr.first].merge(pr.second) || true) work.push_back(pr.first);
    }
    while (!work.empty()) {
      Item it = work.back();
      work.pop_back();
      int p = ip(it), d = id(it);
      if (d >= (int)G.rhs[p].size() || !G.is_nt(G.rhs[p][d])) continue;
      Bits look;
      first_of_seq(p, d + 1, la[it], look);
      for (int q : G.prods_of[G.rhs[p][d] - T]) {
        Item ni = mk(q, 0);
        bool fresh = !la.count(ni);
        if (la[ni].merge(look) || fresh) work.push_back(ni);
      }
    }
    return la;
  };

  // lookahead determination for kernel items
  std::vector<std::map<Item, Bits>> kla(NS);
  std::vector<std::map<Item, std::vector<std::pair<int, Item>>>> prop(NS);
  for (int s = 0; s < NS; ++s)
    for (Item k : kernels[s]) kla[s][k];
  {
    Bits e;
    e.set(T);
    kla[0][mk(0, 0)].merge(e);
  }
  for (int s = 0; s < NS; ++s) {
    for (Item k : kernels[s]) {
      Bits probe;
      probe.set(PROBE);
      auto J = closure1({{k, probe}});
      for (auto& jt : J) {
        int p = ip(jt.first), d = id(jt.first);
        if (d >= (int)G.rhs[p].size()) continue;
        int X = G.rhs[p][d];
        int tgt = edges[s].at(X);
        Item moved = mk(p, d + 1);
        Bits spont = jt.second;
        if (spont.test(PROBE)) {
          prop[s][k].push_back({tgt, moved});
          spont.w[PROBE >> 6] &= ~(1ull << (PROBE & 63));
        }
        kla[tgt][moved].merge(spont);
      }
    }
  }
  for (bool ch = true; ch;) {
    ch = false;
    for (int s = 0; s < NS; ++s)
      for (auto& pk : prop[s]) {
        const Bits src = kla[s][pk.first];
        for (auto& dst : pk.second) ch |= kla[dst.first][dst.second].merge(src);
      }
  }

  // tables
  out.T = T;
  out.N = G.N - 1;  // S' has no GOTO column
  out.n_states = NS;
  out.action.assign((size_t)NS * (T + 1), 0);
  out.go.assign((size_t)NS * std::max(out.N, 1), kNoGoto);
  out.prod.resize(P);
  for (int p = 0; p < P; ++p) out.prod[p] = (uint32_t)G.lhs[p] | (uint32_t)G.rhs[p].size() << 16;
  auto sym_name = [&](int x) -> std::string {
    if (x == T) return "$end";
    return x < T ? g.terminals[x].name : "<nonterminal>";
  };
  auto conflict = [&](int s, int t, uint16_t a, uint16_t b) {
    auto describe = [&](uint16_t v) -> std::string {
      if ((v & 0xC000) == kActShift) return "shift";
      if ((v & 0xC000) == kActAccept) return "accept";
      int p = v & 0x3FFF;
      std::string r = "reduce rule " + std::to_string(p) + " (";
      for (int x : G.rhs[p]) r += (G.is_nt(x) ? std::string("nt") : sym_name(x)) + " ";
      return r + ")";
    };
    throw Error(GRID_E_LALR_CONFLICT, "LALR(1) conflict in state " + std::to_string(s) + " on " +
                                          sym_name(t) + ": " + describe(a) + " vs " + describe(b));
  };
  // completion estimate of every state: the fewest terminals that finish one
  // of its kernel items (the shortest terminal yield of what follows the dot;
  // nonterminals by the least fixpoint of their shortest derivations)
  {
    std::vector<int> minlen(G.N, 1 << 20);
    for (bool ch = true; ch;) {
      ch = false;
      for (int p = 0; p < P; ++p) {
        long sum = 0;
        for (int x : G.rhs[p]) sum += G.is_nt(x) ? minlen[x - T] : 1;
        if (sum < minlen[G.lhs[p]]) {
          minlen[G.lhs[p]] = (int)sum;
          ch = true;
        }
      }
    }
    out.complete_est.assign(NS, 0);
    for (int s = 0; s < NS; ++s) {
      long best = 1 << 20;
      for (auto& kv : kla[s]) {
        const int p = ip(kv.first), d = id(kv.first);
        long sum = 0;
        for (size_t k = (size_t)d; k < G.rhs[p].size(); ++k) {
          const int x = G.rhs[p][k];
          sum += G.is_nt(x) ? minlen[x - T] : 1;
        }
        best = std::min(best, sum);
      }
      out.complete_est[s] = (uint16_t)std::min<long>(best, 0xFFFF);
    }
  }
  out.state_sym.assign(NS, kNoSymbol);
  for (int s = 0; s < NS; ++s) {
    for (auto& e : edges[s]) {
      if (e.first < T) out.action[(size_t)s * (T + 1) + e.first] = (uint16_t)(kActShift | e.second);
      else if (e.first - T < out.N) out.go[(size_t)s * out.N + (e.first - T)] = (uint16_t)e.second;
      // the symbol on which every transition into a state is taken (an LR(0)
      // state has one accessing symbol): terminals by id, nonterminals tagged
      out.state_sym[e.second] = e.first < T ? (uint32_t)e.first : kSymNonterminal | (uint32_t)(e.first - T);
    }
    std::vector<std::pair<Item, Bits>> seed(kla[s].begin(), kla[s].end());
    auto J = closure1(seed);
    for (auto& jt : J) {
      int p = ip(jt.first), d = id(jt.first);
      if (d != (int)G.rhs[p].size()) continue;
      for (int t = 0; t <= T; ++t) {
        if (!jt.second.test(t)) continue;
        uint16_t a = (p == 0) ? kActAccept : (uint16_t)(kActReduce | p);
        uint16_t& cell = out.action[(size_t)s * (T + 1) + t];
        if (cell != 0 && cell != a) conflict(s, t, cell, a);
        cell = a;
      }
    }
  }
  compact_tables(out);
  return out;
}

// The kernels' GOTO.  A unit state (no shift, no GOTO, every action a
// reduction by the same production X -> A with |A| = 1) is reduced the moment
// it is entered: the reduction pops it and takes GOTO(b, X) from the state b
// it was entered from.  So a transition b --A--> unit state is redirected to
// GOTO(b, X), and again while that is a unit state.  A unit state never stays
// on a stack below a shifted terminal, so every stack after a shift is the one
// the LALR tables give; a lookahead the unit state has no action for is
// refused further up the chain (the unit item's lookaheads include everything
// the states reached from b through X can shift or reduce on), so the
// terminals that can be shifted next are the same.
std::vector<int> skip_unit_states(Parser& P) {
  const int NS = P.n_states, T1 = P.T + 1, N = P.N;
  std::vector<int> unit(NS, -1);
  for (int s = 0; s < NS; ++s) {
    int p = -1;
    bool ok = true;
    for (int t = 0; t < T1 && ok; ++t) {
      const uint16_t a = P.act(s, t);
      if (a == 0) continue;
      if ((a & 0xC000) != kActReduce || (p >= 0 && (a & 0x3FFF) != p)) ok = false;
      p = a & 0x3FFF;
    }
    for (int a = 0; a < N && ok; ++a)
      if (P.gto(s, a) != kNoGoto) ok = false;
    if (ok && p > 0 && (P.prod[p] >> 16) == 1) unit[s] = p;
  }
  P.go_skip = P.go;
  for (int b = 0; b < NS; ++b)
    for (int a = 0; a < N; ++a) {
      uint16_t g = P.gto(b, a);
      for (int guard = 0; g != kNoGoto && unit[g] >= 0 && guard <= NS; ++guard) {
        const uint16_t g2 = P.gto(b, (int)(P.prod[unit[g]] & 0xFFFF));
        if (g2 == kNoGoto) break;
        g = g2;
      }
      P.go_skip[(size_t)b * N + a] = g;
    }
  return unit;
}

// Compact tables for simulating a whole set of lookahead terminals at once:
// per state the terminals that shift (or accept, end-of-input column), the
// terminals reduced by the state's main production, and any further reduce
// productions with their own terminal sets; productions appear as
// lhs | length << 16 (empty runs folded in, see below), so a reduce needs no
// further lookup; GOTO (GOTO_SKIP) as an
// open-addressing hash of (key, target) pairs.  Terminal sets take TW words,
// TW a power of two (at least 2), and a state record is padded to a multiple of 16 bytes
// so the kernels read it with 16-byte loads.  The first padding word locates the
// state's shift targets: one u16 per set shift bit, in terminal order, so the target
// of terminal t is entry (number of shift bits below t) of the state's run.
void compact_tables(Parser& P) {
  const std::vector<int> unit = skip_unit_states(P);
  const int T1 = P.T + 1;
  int TW = 2;
  while (TW * 32 < T1) TW *= 2;
  if (TW > kTermWords) throw Error(GRID_E_CAPACITY, "more than 255 terminals");
  P.tw = TW;
  const int stride = parse_record_words(TW);
  P.pstate.assign((size_t)P.n_states * stride, 0);
  P.predx.clear();
  P.pshift.clear();
  // Empty runs: in a state with a reduction by an empty production, the
  // reductions taken on lookahead t up to the first one that pops an entry
  // below the state depend on (state, t) alone -- the empty ones push and pop
  // nothing -- so when that run ends in a reduction X -> alpha popping all k
  // entries it pushed, the run's net effect is one reduction: pop |alpha| - k
  // entries, GOTO on X.  The record keeps that reduction (X | (|alpha| - k) <<
  // 16) for t in place of the first empty one -- one step of a reduce chain
  // instead of k + 1, with the same stack after it -- when every terminal of
  // that empty production's group shares the run.
  auto empty_run = [&](int s0, int t) -> uint32_t {
    int st = s0, k = 0;
    for (int guard = 0; guard <= P.n_states; ++guard) {
      const uint16_t a = P.act(st, t);
      if ((a & 0xC000) != kActReduce) return 0;
      const uint32_t pr = P.prod[a & 0x3FFF];
      const uint32_t len = pr >> 16, X = pr & 0xFFFF;
      if (len == 0) {
        const uint16_t g = P.go_skip[(size_t)st * P.N + X];
        if (g == kNoGoto) return 0;
        st = g;
        ++k;
        continue;
      }
      return k > 0 && len >= (uint32_t)k ? X | (len - (uint32_t)k) << 16 : 0u;
    }
    return 0;
  };
  std::vector<std::pair<uint32_t, uint16_t>> gotos;
  for (int s = 0; s < P.n_states; ++s) {
    uint32_t* rec = &P.pstate[(size_t)s * stride];
    // an empty production's terminals take their run's reduction when they
    // all share one (so the state keeps its number of reduce groups, which is
    // what the set simulation pays for)
    std::map<int, uint32_t> run_of;  // empty production -> the shared run (0 none)
    for (int t = 0; t < T1; ++t) {
      const uint16_t a = P.act(s, t);
      if ((a & 0xC000) != kActReduce || (P.prod[a & 0x3FFF] >> 16) != 0) continue;
      const uint32_t r = empty_run(s, t);
      auto it = run_of.find(a & 0x3FFF);
      if (it == run_of.end()) run_of[a & 0x3FFF] = r;
      else if (it->second != r) it->second = 0;
    }
    std::map<uint32_t, std::vector<uint32_t>> groups;  // reduction (lhs | pops << 16) -> bits
    for (int t = 0; t < T1; ++t) {
      const uint16_t a = P.act(s, t);
      const uint16_t kind = a & 0xC000;
      if (a == 0) continue;
      if (kind == kActShift || kind == kActAccept) {
        rec[t >> 5] |= 1u << (t & 31);
      } else {
        auto it = run_of.find(a & 0x3FFF);
        const uint32_t run = it == run_of.end() ? 0u : it->second;
        auto& g = groups[run ? run : P.prod[a & 0x3FFF]];
        g.resize(TW, 0);
        g[t >> 5] |= 1u << (t & 31);
      }
    }
    uint32_t main_red = 0xFFFFFFFFu;
    size_t best = 0;
    for (auto& g : groups) {
      size_t n = 0;
      for (uint32_t w : g.second) n += (size_t)__builtin_popcount(w);
      if (n > best) { best = n; main_red = g.first; }
    }
    uint32_t n_extra = 0;
    const size_t off = P.predx.size();
    if (off >= (1u << 24)) throw Error(GRID_E_CAPACITY, "reduce groups larger than 2^24 words");
    for (auto& g : groups) {
      if (g.first == main_red) {
        for (int w = 0; w < TW; ++w) rec[TW + w] = g.second[w];
      } else {
        P.predx.push_back(g.first);
        P.predx.insert(P.predx.end(), g.second.begin(), g.second.end());
        ++n_extra;
      }
    }
    if (n_extra > 255) throw Error(GRID_E_CAPACITY, "more than 255 reduce productions in one state");
    rec[2 * TW] = main_red;
    rec[2 * TW + 1] = n_extra | (uint32_t)off << 8;
    rec[2 * TW + 2] = (uint32_t)P.pshift.size();
    for (int t = 0; t < T1; ++t) {
      const uint16_t a = P.act(s, t);
      if ((a & 0xC000) == kActShift) P.pshift.push_back((uint16_t)(a & 0x3FFF));
      else if ((a & 0xC000) == kActAccept) P.pshift.push_back(0);
    }
    // the mask kernels' shift targets: a shift into a unit state (its one
    // reduction pops the shifted entry) goes where that reduction leads, as a
    // GOTO into one does; the stack differs from the LALR one only by that
    // pending reduction, which any lookahead the unit state would accept
    // takes anyway (the device advance keeps the targets above)
    std::vector<uint16_t> red;
    bool moved = false;
    for (int t = 0; t < T1; ++t) {
      const uint16_t a = P.act(s, t);
      if ((a & 0xC000) == kActAccept) red.push_back(0);
      if ((a & 0xC000) != kActShift) continue;
      uint16_t tgt = (uint16_t)(a & 0x3FFF);
      if (unit[tgt] >= 0) {
        const uint16_t g = P.go_skip[(size_t)s * P.N + (P.prod[unit[tgt]] & 0xFFFF)];
        if (g != kNoGoto) {
          tgt = g;
          moved = true;
        }
      }
      red.push_back(tgt);
    }
    rec[2 * TW + 3] = rec[2 * TW + 2];
    if (moved) {
      rec[2 * TW + 3] = (uint32_t)P.pshift.size();
      P.pshift.insert(P.pshift.end(), red.begin(), red.end());
    }
    for (int a = 0; a < P.N; ++a) {
      const uint16_t g = P.go_skip[(size_t)s * P.N + a];
      if (g != kNoGoto) gotos.push_back({goto_key(s, a), g});
    }
  }
  // load factor at most 2/3, so a lookup probes few slots
  int hb = 6;
  while ((size_t)1 << hb < gotos.size() + gotos.size() / 2) ++hb;
  if (P.n_states >= 0xFFFF || P.N > 0xFFFF) throw Error(GRID_E_CAPACITY, "more than 65534 LR states");
  const uint32_t H = 1u << hb;
  P.goto_hbits = hb;
  P.goto_hash.assign((size_t)H * 2, 0);
  for (auto& e : gotos)
    for (uint32_t h = goto_slot(e.first, hb);; h = (h + 1) & (H - 1))
      if (P.goto_hash[2 * h] == 0) {
        P.goto_hash[2 * h] = e.first;
        P.goto_hash[2 * h + 1] = e.second;
        break;
      }
}

}  // namespace grid
