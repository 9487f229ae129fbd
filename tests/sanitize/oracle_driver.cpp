// Runs the oracle (grammar reader, lexicons, vocabulary, viability,
// membership, allowed sets, masks in both modes) on one case file; built
// with AddressSanitizer and UndefinedBehaviorSanitizer by the CPU tests.
#include "../../oracle/oracle.h"
#include "case_reader.h"

int main(int argc, char** argv) {
  Case c;
  if (argc < 2 || !read_case(argv[1], c)) return 2;
  char err[512] = {0};
  void* g = oracle_grammar_new(c.grammar.c_str(), c.drop.c_str(), err, sizeof err);
  if (!g) {
    std::fprintf(stderr, "grammar: %s\n", err);
    return 1;
  }
  void* lex = nullptr;
  if (!c.cat_names.empty()) {
    std::vector<const char*> names, words;
    for (size_t i = 0; i < c.cat_names.size(); ++i) {
      names.push_back(c.cat_names[i].c_str());
      words.push_back(c.cat_words[i].c_str());
    }
    lex = oracle_lexicon_new(g, (int)names.size(), names.data(), words.data(), err, sizeof err);
    if (!lex) {
      std::fprintf(stderr, "lexicon: %s\n", err);
      return 1;
    }
  }
  std::vector<uint8_t> bytes;
  std::vector<uint64_t> off;
  flatten(c.vocab, bytes, off);
  const int V = (int)c.vocab.size();
  void* voc = oracle_vocab_new(bytes.data(), off.data(), V, c.specials.data(), (int)c.specials.size(), c.eos);
  const int T = oracle_num_terminals(g);
  std::vector<uint8_t> allowed(T);
  std::vector<uint32_t> words((V + 31) / 32);
  std::vector<int32_t> ids;
  for (int t = 0; t < V && ids.size() < 64; t += 1 + V / 64) ids.push_back(t);
  std::vector<uint8_t> b0(ids.size()), b1(ids.size());
  int viable = 0, mism = 0, masks = 0;
  for (const auto& w : c.prefixes) {
    const uint8_t* p = (const uint8_t*)w.data();
    viable += oracle_viable(g, lex, p, w.size());
    oracle_member(g, lex, p, w.size());
    oracle_allowed(g, lex, p, w.size(), allowed.data());
    if (masks < c.n_masks && oracle_viable(g, lex, p, w.size())) {
      int32_t e0 = 0, e1 = 0;
      oracle_mask(g, lex, voc, p, w.size(), 1, nullptr, 0, words.data(), nullptr, &e1, 1);
      oracle_mask(g, lex, voc, p, w.size(), 0, ids.data(), (int)ids.size(), nullptr, b0.data(), &e0, 1);
      oracle_mask(g, lex, voc, p, w.size(), 1, ids.data(), (int)ids.size(), nullptr, b1.data(), &e1, 1);
      for (size_t i = 0; i < ids.size(); ++i) mism += b0[i] != b1[i];
      mism += e0 != e1;
      ++masks;
    }
  }
  oracle_vocab_free(voc);
  if (lex) oracle_lexicon_free(lex);
  oracle_grammar_free(g);
  char err2[256];
  const char* bad[] = {"start s\ns : ;", "start s\ntoken A /(/\ns : A ;", "token A \"a\"\n"};
  for (const char* t : bad) {
    void* h = oracle_grammar_new(t, "", err2, sizeof err2);
    if (h) oracle_grammar_free(h);
  }
  std::printf("oracle driver: %d of %zu prefixes viable, %d masks, %d mode mismatches\n", viable, c.prefixes.size(),
              masks, mism);
  return mism ? 1 : 0;
}
