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
// Scan summary (section 4.1: the walk carries the scan state; section 4.2: a
// token either stays inside the current lexeme or crosses boundaries): for
// every DFA state q and spelling u, where maximal munch ends lexemes in u when
// the scan resumes in q, packed as in lexhash.h.  It depends on the lexer and
// the vocabulary only, so it is built once per compile.
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
  for (size_t u = 0; u < U; ++u)
    for (uint32_t k = va.alias_off[u]; k < va.alias_off[u + 1]; ++k) va.spell_of_id[va.alias_ids[k]] = (uint32_t)u;
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

std::vector<uint32_t> build_scan_summary(const LexerDfa& dfa, const VocabArtifacts& va) {
  const size_t U = va.spell_off.size() - 1;
  if ((uint32_t)dfa.S > kScanMaxStates || U == 0) return {};
  std::vector<uint32_t> out((size_t)dfa.S * U);
  auto one = [&](int q, size_t u) -> uint32_t {
    const uint8_t* b = va.spell_bytes.data() + va.spell_off[u];
    const uint32_t n = va.spell_off[u + 1] - va.spell_off[u];
    uint32_t cur = (uint32_t)q, q_first = 0, p_first = 0, ends = 0;
    for (uint32_t i = 0; i < n; ++i) {
      const uint32_t nq = dfa.step((int)cur, b[i]);
      if (nq != (uint32_t)kDead) {
        cur = nq;
        continue;
      }
      // byte i ends the lexeme in state cur; it must accept something, and
      // byte i must start the next lexeme
      if (!dfa.accepting[cur]) return kScanReject;
      if (ends == 0) {
        q_first = cur;
        p_first = i;
      }
      if (++ends == 2) return scan_word(0, q_first, p_first, 2);
      cur = dfa.step(kStart, b[i]);
      if (cur == (uint32_t)kDead) return kScanReject;
    }
    return scan_word(cur, q_first, p_first, ends);
  };
  const int nt = (int)std::max(1u, std::min(16u, std::thread::hardware_concurrency()));
  std::vector<std::thread> pool;
  for (int w = 0; w < nt; ++w)
    pool.emplace_back([&, w]() {
      for (int q = w; q < dfa.S; q += nt)
        for (size_t u = 0; u < U; ++u) out[(size_t)q * U + u] = one(q, u);
    });
  for (auto& th : pool) th.join();
  return out;
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

void add_lexicon(LexiconStore& st, const LexerDfa& dfa, const GrammarText& g,
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
  uint32_t rec[kSlotWords] = {flags_base, hash_base, size - 1, restricted, (uint32_t)nodes.size(),
                              pref_base,  psize - 1, 0};
  st.slots.insert(st.slots.end(), rec, rec + kSlotWords);
  st.n_slots += 1;
}

}  // namespace grid
