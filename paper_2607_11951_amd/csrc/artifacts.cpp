// artifacts.cpp -- vocabulary and schema-lexicon artifacts.
//
// Vocabulary (Definition 3, section 4.1): the distinct non-special spellings,
// sorted in byte order (the depth-first order of the token byte trie), each
// with a 16-byte record (first 8 bytes, first id, length) and a 16-byte
// tail chunk (bytes 8..23) at the same index, longer spellings continuing in
// overflow chunks, so a walk fetches 16 bytes per load;
// an alias table lists every token id sharing a spelling (section 2: masks are
// over ids, so alias expansion is needed for completeness); and a levelized
// CSR form of the same trie (level by level, children in byte order, each
// node pointing at its parent and at the spelling that ends there).
//
// Lexeme-program classes (section 4.1: the walk carries the scan state;
// section 4.2: a token either stays inside the current lexeme or crosses
// boundaries, and tokens with equal verdict inputs form classes): for every
// DFA state q and token id, the class of its lexeme program from q, laid out
// as in lexhash.h.  It depends on the lexer and the vocabulary only, so it is
// built once per compile.
//
// Schema lexicon (section 2, L3): per slot, one byte trie over the words of
// every category with per-node flags "prefix of a category-c word" and
// "category-c word", edges in a hash table and the nodes of depth 1..8 in a
// prefix table keyed by their bytes (lexhash.h).  Each word must be a
// lexeme of its category's terminal (W_c subset of R_c, Proposition 8 (d)).
#include <algorithm>
#include <cstring>
#include <map>
#include <numeric>
#include <thread>
#include <unordered_map>

#include "host.h"
#include "lexhash.h"

namespace grid {

VocabArtifacts build_vocab(const uint8_t* bytes, const uint64_t* off, int V, const int32_t* specials,
                           int n_special, int eos_id) {
  if (V < 1) throw Error(GRID_E_VOCAB, "vocabulary is empty");
  if (!off || (!bytes && off[V] != 0)) throw Error(GRID_E_ARG, "vocabulary pointers are null");
  for (int t = 0; t < V; ++t)
    if (off[t + 1] < off[t]) throw Error(GRID_E_VOCAB, "vocabulary offsets decrease at id " + std::to_string(t));
  if (eos_id < -1 || eos_id >= V) throw Error(GRID_E_ARG, "eos_id out of range");
  std::vector<char> special(V, 0);
  for (int k = 0; k < n_special; ++k) {
    if (specials[k] < 0 || specials[k] >= V) throw Error(GRID_E_ARG, "special id out of range");
    special[specials[k]] = 1;
  }
  if (eos_id >= 0) special[eos_id] = 1;
  VocabArtifacts va;
  va.V = V;
  va.eos_id = eos_id;
  std::vector<int> ids;
  for (int t = 0; t < V; ++t) {
    uint64_t len = off[t + 1] - off[t];
    if (special[t] || len == 0) continue;
    if (len > 255) throw Error(GRID_E_CAPACITY, "token " + std::to_string(t) + " is longer than 255 bytes");
    ids.push_back(t);
  }
  auto spell = [&](int t) {
    return std::string((const char*)bytes + off[t], (size_t)(off[t + 1] - off[t]));
  };
  // byte order (the depth-first order of the token trie): the 64 spellings a
  // wave walks together share prefixes, so their lanes tend to stop together
  std::stable_sort(ids.begin(), ids.end(), [&](int a, int b) {
    size_t la = off[a + 1] - off[a], lb = off[b + 1] - off[b];
    int c = memcmp(bytes + off[a], bytes + off[b], std::min(la, lb));
    return c != 0 ? c < 0 : la < lb;
  });
  va.spell_off.push_back(0);
  va.alias_off.push_back(0);
  std::vector<std::string> uniq;
  for (size_t k = 0; k < ids.size(); ++k) {
    std::string s = spell(ids[k]);
    if (uniq.empty() || uniq.back() != s) {
      if (!uniq.empty()) va.alias_off.push_back((uint32_t)va.alias_ids.size());
      uniq.push_back(s);
      va.spell_bytes.insert(va.spell_bytes.end(), s.begin(), s.end());
      va.spell_off.push_back((uint32_t)va.spell_bytes.size());
      va.max_len = std::max(va.max_len, (int)s.size());
      uint64_t head = 0;
      for (size_t k = 0; k < s.size() && k < 8; ++k) head |= (uint64_t)(uint8_t)s[k] << (8 * k);
      va.spell_rec.push_back((uint32_t)head);
      va.spell_rec.push_back((uint32_t)(head >> 32));
      va.spell_rec.push_back((uint32_t)ids[k]);
      va.spell_rec.push_back((uint32_t)s.size());  // | overflow chunk << 8, below
    } else {
      va.spell_rec[va.spell_rec.size() - 2] |= 1u << 31;  // more than one id
    }
    va.alias_ids.push_back(ids[k]);
  }
  if (!uniq.empty()) va.alias_off.push_back((uint32_t)va.alias_ids.size());
  va.spell_bytes.resize(va.spell_bytes.size() + 32, 0);  // safe over-read padding
  // tails: chunk u holds bytes 8..23 of spelling u, so it can be fetched with
  // the record; bytes 24.. of longer spellings follow in overflow chunks
  const size_t U = uniq.size();
  va.spell_tail.assign(U * 16, 0);
  for (size_t u = 0; u < U; ++u) {
    const std::string& sp = uniq[u];
    for (size_t k = 8; k < sp.size() && k < 24; ++k) va.spell_tail[u * 16 + k - 8] = (uint8_t)sp[k];
    if (sp.size() > 24) {
      const size_t chunk = va.spell_tail.size() / 16;
      if (chunk >= (1u << 24)) throw Error(GRID_E_CAPACITY, "spelling tails larger than 256 MiB");
      va.spell_tail.insert(va.spell_tail.end(), sp.begin() + 24, sp.end());
      va.spell_tail.resize((va.spell_tail.size() + 15) & ~(size_t)15, 0);
      va.spell_rec[u * 4 + 3] |= (uint32_t)chunk << 8;
    }
  }
  va.spell_tail.resize(va.spell_tail.size() + 32, 0);  // read-ahead padding
  std::vector<char> single(256, 0);
  for (auto& s : uniq)
    if (s.size() == 1) single[(uint8_t)s[0]] = 1;
  va.byte_complete = std::all_of(single.begin(), single.end(), [](char c) { return c != 0; });
  va.spell_of_id.assign(V, 0xFFFFFFFFu);
  va.id_first.assign(V, 0);
  va.id_head.assign(V, 0);
  for (size_t u = 0; u < U; ++u)
    for (uint32_t k = va.alias_off[u]; k < va.alias_off[u + 1]; ++k) {
      va.spell_of_id[va.alias_ids[k]] = (uint32_t)u;
      va.id_first[va.alias_ids[k]] = (uint8_t)uniq[u][0];
      va.id_head[va.alias_ids[k]] =
          (uint8_t)uniq[u][0] | (uniq[u].size() > 1 ? 0x10000u | (uint32_t)(uint8_t)uniq[u][1] << 8 : 0u);
    }
  // first-byte range of every 64 consecutive spellings (first bytes are
  // non-decreasing, so the first and the last spelling of the group bound it)
  for (size_t u0 = 0; u0 < uniq.size(); u0 += 64) {
    const size_t u1 = std::min(uniq.size(), u0 + 64) - 1;
    va.sub_range.push_back((uint16_t)((uint8_t)uniq[u0][0] | (uint8_t)uniq[u1][0] << 8));
  }

  // levelized trie: nodes of level L are the distinct length-L prefixes,
  // ordered by (parent, byte) -- the byte order of the prefixes themselves
  std::vector<std::vector<std::pair<std::string, int>>> levels(va.max_len + 1);
  for (size_t u = 0; u < uniq.size(); ++u)
    for (size_t L = 1; L <= uniq[u].size(); ++L) {
      auto& lv = levels[L];
      std::string p = uniq[u].substr(0, L);
      if (lv.empty() || lv.back().first != p) lv.push_back({p, -1});
      if (L == uniq[u].size()) lv.back().second = (int)u;
    }
  va.level_off.assign(va.max_len + 2, 0);
  std::map<std::string, uint32_t> index_of;  // prefix -> global node index
  uint32_t next = 0;
  for (int L = 1; L <= va.max_len; ++L) {
    va.level_off[L - 1] = next;
    for (auto& pr : levels[L]) {
      uint32_t parent = 0;
      if (L > 1) parent = index_of.at(pr.first.substr(0, L - 1)) + 1;
      if (parent >= (1u << 24)) throw Error(GRID_E_CAPACITY, "trie larger than 2^24 nodes");
      va.trie_nodes.push_back((uint8_t)pr.first.back() | parent << 8);
      va.trie_nodes.push_back((uint32_t)(pr.second + 1));
      index_of[pr.first] = next++;
    }
  }
  va.level_off[va.max_len] = next;
  va.level_off[va.max_len + 1] = next;
  return va;
}

ClassTables build_class_tables(const LexerDfa& dfa, const VocabArtifacts& va) {
  const size_t U = va.spell_off.size() - 1;
  const size_t S = (size_t)dfa.S, V = (size_t)va.V;
  if (S * V > ((size_t)3 << 29))
    throw Error(GRID_E_CAPACITY, "class map of " + std::to_string(S) + " lexer states x " + std::to_string(V) +
                                     " tokens is larger than 3 GiB");
  ClassTables ct;
  ct.map.assign(S * V, 0);
  std::vector<std::vector<uint32_t>> recs(S);
  // the lexeme program of spelling u when the scan resumes in q
  auto program = [&](uint32_t q, size_t u, uint32_t (&r)[4]) {
    const uint8_t* b = va.spell_bytes.data() + va.spell_off[u];
    const uint32_t n = va.spell_off[u + 1] - va.spell_off[u];
    uint32_t cur = q, ends = 0, qe[kClassEnds] = {0, 0, 0}, pe[kClassEnds] = {0, 0, 0}, flags = 0;
    for (uint32_t i = 0; i < n; ++i) {
      const uint32_t nq = dfa.step((int)cur, b[i]);
      if (nq != (uint32_t)kDead) {
        cur = nq;
        continue;
      }
      // byte i ends the lexeme in state cur; it must accept something, and
      // byte i must start the next lexeme
      if (!dfa.accepting[cur]) {
        r[0] = kClassReject, r[1] = r[2] = r[3] = 0;
        return;
      }
      if (i == 0) flags |= kClassP0;
      if (ends < (uint32_t)kClassEnds) {
        qe[ends] = cur;
        pe[ends] = i;
      }
      ++ends;
      cur = dfa.step(kStart, b[i]);
      if (cur == (uint32_t)kDead) {
        r[0] = kClassReject, r[1] = r[2] = r[3] = 0;
        return;
      }
    }
    r[0] = (ends > (uint32_t)kClassEnds ? kClassMore : ends) | flags;
    r[1] = cur | qe[0] << 16;
    r[2] = qe[1] | qe[2] << 16;
    r[3] = pe[0] | pe[1] << 8 | pe[2] << 16;
  };
  struct Key {
    uint32_t a, b, c, d;
    bool operator==(const Key& o) const { return a == o.a && b == o.b && c == o.c && d == o.d; }
  };
  struct KeyHash {
    size_t operator()(const Key& k) const {
      uint64_t h = ((uint64_t)k.a << 32 | k.b) * 0x9E3779B97F4A7C15ull ^
                   ((uint64_t)k.c << 32 | k.d) * 0xC2B2AE3D27D4EB4Full;
      return (size_t)(h ^ (h >> 29));
    }
  };
  const int nt = (int)std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  std::vector<std::thread> pool;
  for (int w = 0; w < nt; ++w)
    pool.emplace_back([&, w]() {
      std::vector<uint16_t> local(U);
      std::unordered_map<Key, uint32_t, KeyHash> seen;
      for (size_t q = (size_t)w; q < S; q += (size_t)nt) {
        seen.clear();
        std::vector<uint32_t>& rq = recs[q];
        rq = {kClassReject, 0, 0, 0, kClassWalk, 0, 0, 0};  // local classes 0 and 1
        for (size_t u = 0; u < U; ++u) {
          uint32_t r[4];
          program((uint32_t)q, u, r);
          if (r[0] & kClassReject) {
            local[u] = 0;
            continue;
          }
          auto it = seen.find(Key{r[0], r[1], r[2], r[3]});
          if (it != seen.end()) {
            local[u] = (uint16_t)it->second;
            continue;
          }
          const uint32_t c = (uint32_t)(rq.size() / 4);
          if (c >= kClassMaxLocal) {  // beyond capacity: this token walks its bytes
            local[u] = 1;
            continue;
          }
          seen.emplace(Key{r[0], r[1], r[2], r[3]}, c);
          rq.insert(rq.end(), {r[0], r[1], r[2], r[3]});
          local[u] = (uint16_t)c;
        }
        uint16_t* m = ct.map.data() + q * V;
        for (size_t id = 0; id < V; ++id) {
          const uint32_t u = va.spell_of_id[id];
          m[id] = u == 0xFFFFFFFFu ? (uint16_t)0 : local[u];
        }
      }
    });
  for (auto& th : pool) th.join();
  ct.off.assign(S + 1, 0);
  for (size_t q = 0; q < S; ++q) {
    ct.off[q + 1] = ct.off[q] + (uint32_t)(recs[q].size() / 4);
    ct.max_classes = std::max(ct.max_classes, ct.off[q + 1] - ct.off[q]);
  }
  ct.rec.reserve((size_t)ct.off[S] * 4);
  for (size_t q = 0; q < S; ++q) ct.rec.insert(ct.rec.end(), recs[q].begin(), recs[q].end());
  return ct;
}

uint32_t LexiconStore::child(int slot, uint32_t node, uint8_t b) const {
  if (node == kNoLex) return kNoLex;
  const uint32_t* sl = &slots[(size_t)slot * kSlotWords];
  uint32_t key = lex_key(node, b), mask = sl[2];
  for (uint32_t h = lex_hash(key) & mask;; h = (h + 1) & mask) {
    const uint32_t* e = &hash[(size_t)(sl[1] + h) * 2];
    if (e[0] == key) return e[1];
    if (e[0] == 0) return kNoLex;
  }
}

uint16_t LexiconStore::node_flags(int slot, uint32_t node) const {
  if (node == kNoLex) return 0;
  return flags[slots[(size_t)slot * kSlotWords] + node];
}

void add_lexicon(LexiconStore& st, const LexerDfa& dfa, const GrammarText& g, const VocabArtifacts& va,
                 const std::vector<int>& term_cat,
                 const std::vector<std::pair<std::string, std::vector<std::string>>>& cats) {
  struct Node {
    uint16_t flags = 0;
    std::map<uint8_t, uint32_t> kids;
  };
  std::vector<Node> nodes(1);
  uint32_t restricted = 0;
  for (auto& cw : cats) {
    int t = -1;
    for (size_t k = 0; k < g.terminals.size(); ++k)
      if (g.terminals[k].name == cw.first) t = (int)k;
    if (t < 0 || term_cat[t] < 0)
      throw Error(GRID_E_ARG, "lexicon category '" + cw.first + "' is not a category terminal");
    int c = term_cat[t];
    restricted |= 1u << c;
    nodes[0].flags |= (uint16_t)(1u << c);
    for (const std::string& w : cw.second) {
      if (w.empty()) continue;
      // W_c must be inside R_c: the DFA accepts the word as terminal t
      int q = kStart;
      for (unsigned char ch : w) {
        q = dfa.step(q, ch);
        if (q == kDead) break;
      }
      bool ok = false;
      if (q != kDead)
        for (uint32_t k = dfa.accept_off[q]; k < dfa.accept_off[q + 1]; ++k) ok |= dfa.accept_list[k] == t;
      if (!ok)
        throw Error(GRID_E_LEXICON, "lexicon word '" + w + "' is not a lexeme of " + cw.first);
      uint32_t n = 0;
      for (unsigned char ch : w) {
        auto it = nodes[n].kids.find(ch);
        uint32_t nx;
        if (it == nodes[n].kids.end()) {
          nx = (uint32_t)nodes.size();
          nodes[n].kids[ch] = nx;
          nodes.emplace_back();
        } else {
          nx = it->second;
        }
        n = nx;
        nodes[n].flags |= (uint16_t)(1u << c);
      }
      nodes[n].flags |= (uint16_t)(1u << (8 + c));
    }
  }
  if (nodes.size() >= (1u << 24)) throw Error(GRID_E_CAPACITY, "lexicon trie larger than 2^24 nodes");
  size_t n_edges = nodes.size() - 1;
  uint32_t size = 1;
  while (size < 2 * n_edges + 1) size <<= 1;
  uint32_t flags_base = (uint32_t)st.flags.size();
  uint32_t hash_base = (uint32_t)(st.hash.size() / 2);
  st.flags.resize(st.flags.size() + nodes.size());
  for (size_t k = 0; k < nodes.size(); ++k) st.flags[flags_base + k] = nodes[k].flags;
  st.child_bits.resize(st.flags.size() * 8, 0u);
  for (size_t k = 0; k < nodes.size(); ++k)
    for (auto& e : nodes[k].kids) st.child_bits[(flags_base + k) * 8 + (e.first >> 5)] |= 1u << (e.first & 31u);
  st.hash.resize(st.hash.size() + (size_t)size * 2, 0);
  for (size_t k = 0; k < nodes.size(); ++k)
    for (auto& e : nodes[k].kids) {
      uint32_t key = lex_key((uint32_t)k, e.first);
      for (uint32_t h = lex_hash(key) & (size - 1);; h = (h + 1) & (size - 1)) {
        uint32_t* slot = &st.hash[(size_t)(hash_base + h) * 2];
        if (slot[0] == 0) {
          slot[0] = key;
          slot[1] = e.second;
          break;
        }
      }
    }
  // prefix table: every node of depth 1..8 keyed by its bytes
  std::vector<std::pair<uint64_t, uint32_t>> pref;  // (bytes, len << 24 | node)
  {
    std::vector<std::pair<uint32_t, std::pair<uint64_t, uint32_t>>> todo{{0u, {0ull, 0u}}};
    while (!todo.empty()) {
      auto [n, kb] = todo.back();
      todo.pop_back();
      if (kb.second >= 8) continue;
      for (auto& e : nodes[n].kids) {
        const uint64_t b2 = kb.first | (uint64_t)e.first << (8 * kb.second);
        pref.push_back({b2, (kb.second + 1) << 24 | e.second});
        todo.push_back({e.second, {b2, kb.second + 1}});
      }
    }
  }
  uint32_t psize = 16;
  while (psize < 2 * pref.size()) psize <<= 1;
  const uint32_t pref_base = (uint32_t)(st.prefix.size() / 4);
  st.prefix.resize(st.prefix.size() + (size_t)psize * 4, 0);
  for (auto& e : pref) {
    const uint32_t lo = (uint32_t)e.first, hi = (uint32_t)(e.first >> 32), len = e.second >> 24;
    const uint32_t node = e.second & 0xFFFFFF;
    for (uint32_t h = lexp_hash(lo, hi, len) & (psize - 1);; h = (h + 1) & (psize - 1)) {
      uint32_t* slot = &st.prefix[(size_t)(pref_base + h) * 4];
      if ((slot[2] & 0xFFFF) == 0) {
        slot[0] = lo;
        slot[1] = hi;
        slot[2] = len | (uint32_t)nodes[node].flags << 16;
        slot[3] = node;
        break;
      }
    }
  }
  // stride table: every node of depth > 8 keyed by its ancestor at the last
  // multiple of 8 above it and its bytes below that ancestor
  struct Deep {
    uint32_t anc, lo, hi, len, node;
  };
  std::vector<Deep> deep;
  {
    struct Todo {
      uint32_t n, depth, anc;
      uint64_t bytes;  // bytes below anc
    };
    std::vector<Todo> todo{{0u, 0u, 0u, 0ull}};
    while (!todo.empty()) {
      const Todo t = todo.back();
      todo.pop_back();
      for (auto& e : nodes[t.n].kids) {
        const uint32_t d = t.depth + 1, k = (d - 1) & 7u;  // k: index of this byte below anc
        const uint64_t b2 = (k == 0 ? 0ull : t.bytes) | (uint64_t)e.first << (8 * k);
        if (d > 8) deep.push_back({t.anc, (uint32_t)b2, (uint32_t)(b2 >> 32), k + 1, e.second});
        // the children of a node at a multiple of 8 hang below it
        todo.push_back({e.second, d, d % 8 == 0 ? e.second : t.anc, b2});
      }
    }
  }
  uint32_t ssize = 16;
  while (ssize < 2 * deep.size()) ssize <<= 1;
  const uint32_t stride_base = (uint32_t)(st.stride.size() / 8);
  st.stride.resize(st.stride.size() + (size_t)ssize * 8, 0);
  for (auto& e : deep) {
    for (uint32_t h = lexs_hash(e.anc, e.lo, e.hi, e.len) & (ssize - 1);; h = (h + 1) & (ssize - 1)) {
      uint32_t* slot = &st.stride[(size_t)(stride_base + h) * 8];
      if ((slot[3] & 0xFFFF) == 0) {
        slot[0] = e.anc;
        slot[1] = e.lo;
        slot[2] = e.hi;
        slot[3] = e.len | (uint32_t)nodes[e.node].flags << 16;
        slot[4] = e.node;
        break;
      }
    }
  }
  // token flags: for every token id and start offset o in {0, 1}, the
  // prefix flags of the token's bytes from o to its end and the word flags of
  // the first lexeme maximal munch cuts from o (scanning from the start state)
  const size_t tok_base = st.token.size();
  st.token.resize(tok_base + (size_t)va.V, 0u);
  st.toksum.resize(tok_base + (size_t)va.V, 0u);
  if (restricted) {
    const size_t U = va.spell_off.size() - 1;
    for (size_t u = 0; u < U; ++u) {
      const uint8_t* b = va.spell_bytes.data() + va.spell_off[u];
      const uint32_t n = va.spell_off[u + 1] - va.spell_off[u];
      uint32_t f = 0;
      for (uint32_t o = 0; o < 2 && o < n; ++o) {
        uint32_t e1 = n, q = kStart;  // end of the first lexeme from o
        for (uint32_t i = o; i < n; ++i) {
          q = dfa.step((int)q, b[i]);
          if (q == (uint32_t)kDead) {
            e1 = i;
            break;
          }
        }
        uint32_t node = 0, pre = 0, word = 0;
        for (uint32_t i = o; i < n; ++i) {
          auto it = nodes[node].kids.find(b[i]);
          if (it == nodes[node].kids.end()) break;
          node = it->second;
          if (i + 1 == e1 && e1 < n) word = nodes[node].flags >> 8;
          if (i + 1 == n) pre = nodes[node].flags & 0xFFu;
        }
        f |= (pre | word << 8) << (16 * o);
      }
      uint8_t sum = 0;  // bit 2o: prefix flags from o nonzero; bit 2o + 1: word flags from o nonzero
      for (int o = 0; o < 2; ++o)
        for (int k = 0; k < 2; ++k)
          if ((f >> (16 * o + 8 * k)) & 0xFFu) sum |= (uint8_t)(1u << (2 * o + k));
      for (uint32_t k = va.alias_off[u]; k < va.alias_off[u + 1]; ++k) {
        st.token[tok_base + va.alias_ids[k]] = f;
        st.toksum[tok_base + va.alias_ids[k]] = sum;
      }
    }
  }
  // the schema fingerprint: FNV-1a over the restricted categories and their
  // sorted word lists, so equal lexicons in any slot or handle share it
  uint32_t schema_fp = 2166136261u;
  auto mix = [&schema_fp](uint32_t v) {
    for (int k = 0; k < 4; ++k) schema_fp = (schema_fp ^ ((v >> (8 * k)) & 0xFFu)) * 16777619u;
  };
  {
    std::vector<std::pair<int, std::vector<std::string>>> by_cat;
    for (auto& cw : cats) {
      int t = -1;
      for (size_t k = 0; k < g.terminals.size(); ++k)
        if (g.terminals[k].name == cw.first) t = (int)k;
      std::vector<std::string> ws(cw.second.begin(), cw.second.end());
      ws.erase(std::remove(ws.begin(), ws.end(), std::string()), ws.end());
      std::sort(ws.begin(), ws.end());
      ws.erase(std::unique(ws.begin(), ws.end()), ws.end());
      by_cat.push_back({term_cat[t], ws});
    }
    std::sort(by_cat.begin(), by_cat.end());
    for (auto& cw : by_cat) {
      mix(0xC0DE0000u | (uint32_t)cw.first);
      for (auto& w : cw.second) {
        mix((uint32_t)w.size());
        for (unsigned char ch : w) mix(ch);
      }
    }
  }
  uint32_t rec[kSlotWords] = {flags_base, hash_base, size - 1, restricted, (uint32_t)nodes.size(),
                              pref_base,  psize - 1, stride_base, ssize - 1, schema_fp, 0, 0};
  st.slots.insert(st.slots.end(), rec, rec + kSlotWords);
  st.shortest.resize((size_t)(st.n_slots + 1) * kMaxCategories);
  for (auto& cw : cats) {
    int t = -1;
    for (size_t k = 0; k < g.terminals.size(); ++k)
      if (g.terminals[k].name == cw.first) t = (int)k;
    std::vector<std::string> ws;
    for (const std::string& x : cw.second)
      if (!x.empty()) ws.push_back(x);
    std::sort(ws.begin(), ws.end(), [](const std::string& a, const std::string& b) {
      return a.size() != b.size() ? a.size() < b.size() : a < b;
    });
    ws.erase(std::unique(ws.begin(), ws.end()), ws.end());
    if (ws.size() > 6) ws.resize(6);
    st.shortest[(size_t)st.n_slots * kMaxCategories + (size_t)term_cat[t]] = ws;
  }
  st.n_slots += 1;
}

}  // namespace grid
