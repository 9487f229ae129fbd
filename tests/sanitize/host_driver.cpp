// Runs the library's host C++ (compile, lexicon slots, artifacts, host
// advance, rolling hash, completion writer, error paths) on one case file;
// built with AddressSanitizer and UndefinedBehaviorSanitizer by the CPU tests.
// The device side is not linked: the one host symbol it provides is defined
// here.
#include <cstring>

#include "../../include/grid.h"
#include "case_reader.h"

namespace grid {
int overlay_capacity() { return 16; }
}  // namespace grid

static int fails = 0;
static void expect(bool ok, const char* what) {
  if (!ok) {
    std::fprintf(stderr, "FAILED: %s (%s)\n", what, grid_last_error());
    ++fails;
  }
}

int main(int argc, char** argv) {
  Case c;
  if (argc < 2 || !read_case(argv[1], c)) return 2;
  std::vector<uint8_t> bytes;
  std::vector<uint64_t> off;
  flatten(c.vocab, bytes, off);
  grid_compile_args a{};
  a.grammar = c.grammar.c_str();
  a.grammar_len = c.grammar.size();
  a.drop_labels = c.drop.empty() ? nullptr : c.drop.c_str();
  a.vocab_bytes = bytes.data();
  a.vocab_offsets = off.data();
  a.vocab_size = (int32_t)c.vocab.size();
  a.special_ids = c.specials.data();
  a.n_special = (int32_t)c.specials.size();
  a.eos_id = c.eos;
  grid_compiled* g = nullptr;
  expect(grid_compile(&a, &g) == GRID_OK, "grid_compile");
  if (!g) return 1;
  int32_t slot = 0;
  if (!c.cat_names.empty()) {
    std::vector<const char*> names, words;
    for (size_t i = 0; i < c.cat_names.size(); ++i) {
      names.push_back(c.cat_names[i].c_str());
      words.push_back(c.cat_words[i].c_str());
    }
    grid_lexicon_args la{(int32_t)names.size(), names.data(), words.data()};
    expect(grid_add_lexicon(g, &la, &slot) == GRID_OK, "grid_add_lexicon");
    const char* bad_name = "NO_SUCH_CATEGORY";
    const char* bad_words = "x";
    grid_lexicon_args bad{1, &bad_name, &bad_words};
    int32_t s2 = -1;
    expect(grid_add_lexicon(g, &bad, &s2) != GRID_OK, "unknown category refused");
  }
  grid_info_t info;
  expect(grid_info(g, &info) == GRID_OK, "grid_info");
  uint64_t sum = 0;
  for (int k = 0; k < GRID_ART_COUNT; ++k) {  // every artifact byte is read
    const void* p = nullptr;
    size_t n = 0;
    if (grid_artifact(g, k, &p, &n) != GRID_OK) continue;
    for (size_t i = 0; i < n; ++i) sum += ((const uint8_t*)p)[i];
  }
  std::vector<uint16_t> stack(1 << 16);
  std::vector<uint64_t> hashes(stack.size());
  std::vector<int32_t> toks(4096);
  size_t n_ok = 0;
  for (const auto& w : c.prefixes) {
    grid_config cfg;
    uint32_t depth = 0;
    const int rc = grid_config_from_prefix(g, slot, (const uint8_t*)w.data(), w.size(), &cfg, stack.data(),
                                           (uint32_t)stack.size(), &depth);
    if (rc != GRID_OK) continue;
    ++n_ok;
    expect(grid_stack_hash_host(g, stack.data(), depth, hashes.data()) == GRID_OK, "grid_stack_hash_host");
    int32_t n = 0;
    const int rc2 = grid_complete(g, slot, (const uint8_t*)w.data(), w.size(), (int32_t)toks.size(), toks.data(), &n);
    expect(rc2 == GRID_OK || rc2 == GRID_E_CAPACITY, "grid_complete");
    // a prefix with control bytes appended: completed exactly when it is viable
    std::string odd = w + "\x01\x02\x03";
    grid_config c2;
    const bool viable = grid_config_from_prefix(g, slot, (const uint8_t*)odd.data(), odd.size(), &c2, stack.data(),
                                                (uint32_t)stack.size(), &depth) == GRID_OK;
    const int rc3 = grid_complete(g, slot, (const uint8_t*)odd.data(), odd.size(), (int32_t)toks.size(), toks.data(),
                                  &n);
    expect(viable ? rc3 == GRID_OK || rc3 == GRID_E_CAPACITY : rc3 == GRID_E_NOT_VIABLE,
           "completion refused exactly for non-viable prefixes");
  }
  expect(n_ok > 0, "some prefix is viable");
  grid_free(g);
  // error paths of the compiler
  const char* bad_grammars[] = {"start s\ns : ;", "start s\ntoken A \"a\"\ns : A B ;", "start s\ntoken A /(/\ns : A ;",
                                "token A \"a\"\n", "start s\ntoken A \"a\"\ns : A | A ;"};
  for (const char* t : bad_grammars) {
    grid_compile_args b = a;
    b.grammar = t;
    b.grammar_len = std::strlen(t);
    b.drop_labels = nullptr;
    grid_compiled* h = nullptr;
    if (grid_compile(&b, &h) == GRID_OK) grid_free(h);  // either outcome, no memory error
  }
  std::printf("host driver: %zu prefixes viable of %zu, %d artifacts, checksum %llu, %d failures\n", n_ok,
              c.prefixes.size(), (int)GRID_ART_COUNT, (unsigned long long)sum, fails);
  return fails ? 1 : 0;
}
