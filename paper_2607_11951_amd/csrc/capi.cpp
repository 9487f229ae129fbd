// capi.cpp -- host entry points of the C ABI (compile, artifacts, configs).
#include <cstring>
#include <string>

#include "host.h"
#include "lexhash.h"
#include "rolling_hash.h"

int host_config_from_prefix(const grid_compiled* g, int slot, const uint8_t* w, size_t n,
                            grid_config* cfg, std::vector<uint16_t>& stack);

namespace {
thread_local std::string g_last_error;
}

namespace grid {
int fail(int code, const std::string& msg) {
  g_last_error = msg;
  return code;
}
void clear_error() { g_last_error.clear(); }
}  // namespace grid

using namespace grid;

extern "C" const char* grid_last_error(void) { return g_last_error.c_str(); }

extern "C" int grid_compile(const grid_compile_args* a, grid_compiled** out) {
  clear_error();
  if (!a || !out || !a->grammar) return fail(GRID_E_ARG, "null argument");
  *out = nullptr;
  try {
    auto g = std::make_unique<grid_compiled>();
    g->gram = parse_grammar(std::string(a->grammar, a->grammar_len));
    std::vector<std::string> drop;
    if (a->drop_labels) {
      std::string cur;
      for (const char* p = a->drop_labels;; ++p) {
        if (*p == ',' || *p == 0) {
          size_t b = cur.find_first_not_of(' '), e = cur.find_last_not_of(' ');
          if (b != std::string::npos) drop.push_back(cur.substr(b, e - b + 1));
          cur.clear();
          if (*p == 0) break;
        } else {
          cur += *p;
        }
      }
    }
    g->parser = build_parser(g->gram, drop);
    g->dfa = build_lexer(g->gram);
    const int T = (int)g->gram.terminals.size();
    g->term_cat.assign(T, -1);
    g->term_info.assign(T, 0);
    for (int t = 0; t < T; ++t) {
      const Terminal& tm = g->gram.terminals[t];
      uint32_t info = tm.ignored ? 1u : 0u;
      if (tm.category) {
        if ((int)g->cat_term.size() >= kMaxCategories)
          throw Error(GRID_E_CAPACITY, "more than 8 category terminals");
        g->term_cat[t] = (int)g->cat_term.size();
        g->cat_term.push_back(t);
      }
      info |= (uint32_t)(g->term_cat[t] < 0 ? 0xFF : g->term_cat[t]) << 8;
      g->term_info[t] = info;
    }
    g->vocab = build_vocab(a->vocab_bytes, a->vocab_offsets, a->vocab_size, a->special_ids,
                           a->n_special, a->eos_id);
    g->classes = build_class_tables(g->dfa, g->vocab);
    add_lexicon(g->lex, g->dfa, g->gram, g->vocab, g->term_cat, {});  // slot 0: no restrictions
    // FNV-1a over the tables a cached mask row depends on
    uint32_t fp = 2166136261u;
    auto mix = [&fp](const void* p, size_t n) {
      const uint8_t* b = (const uint8_t*)p;
      for (size_t i = 0; i < n; ++i) fp = (fp ^ b[i]) * 16777619u;
    };
    const int32_t dims[] = {g->dfa.S, g->dfa.C, g->parser.T, g->parser.N, g->parser.n_states, g->vocab.V,
                            (int32_t)g->vocab.spell_off.size()};
    mix(dims, sizeof(dims));
    mix(g->dfa.next.data(), g->dfa.next.size() * 2);
    mix(g->parser.action.data(), g->parser.action.size() * 2);
    mix(g->vocab.spell_bytes.data(), g->vocab.spell_bytes.size());
    mix(g->vocab.alias_ids.data(), g->vocab.alias_ids.size() * 4);
    g->fingerprint = fp;
    // the grammar family's fingerprint: what context-independent words depend
    // on besides the allowed set, the remainder and the lexicon -- the lexer
    // (terminal numbering, priorities, ignored and category flags) and the
    // vocabulary, not the role projection
    uint32_t ff = 2166136261u;
    auto mixf = [&ff](const void* p, size_t n) {
      const uint8_t* b = (const uint8_t*)p;
      for (size_t i = 0; i < n; ++i) ff = (ff ^ b[i]) * 16777619u;
    };
    const int32_t fdims[] = {g->dfa.S, g->dfa.C, T, g->vocab.V, (int32_t)g->vocab.spell_off.size()};
    mixf(fdims, sizeof(fdims));
    mixf(g->dfa.next.data(), g->dfa.next.size() * 2);
    mixf(g->dfa.accept_off.data(), g->dfa.accept_off.size() * 4);
    mixf(g->dfa.accept_list.data(), g->dfa.accept_list.size());
    mixf(g->term_info.data(), g->term_info.size() * 4);
    mixf(g->vocab.spell_bytes.data(), g->vocab.spell_bytes.size());
    mixf(g->vocab.alias_ids.data(), g->vocab.alias_ids.size() * 4);
    g->family_fp = ff;
    *out = g.release();
    return GRID_OK;
  } catch (const Error& e) {
    return fail(e.code, e.what());
  } catch (const std::exception& e) {
    return fail(GRID_E_ARG, e.what());
  }
}

extern "C" void grid_free(grid_compiled* g) { delete g; }

extern "C" int grid_info(const grid_compiled* g, grid_info_t* o) {
  clear_error();
  if (!g || !o) return fail(GRID_E_ARG, "null argument");
  o->n_terminals = g->parser.T;
  o->n_nonterminals = g->parser.N;
  o->n_productions = (int32_t)g->parser.prod.size();
  o->n_lr_states = g->parser.n_states;
  o->n_dfa_states = g->dfa.S;
  o->n_byte_classes = g->dfa.C;
  o->vocab_size = g->vocab.V;
  o->mask_words = (g->vocab.V + 31) / 32;
  o->n_spellings = (int32_t)g->vocab.spell_off.size() - 1;
  o->max_spelling_len = g->vocab.max_len;
  o->n_trie_nodes = (int32_t)(g->vocab.trie_nodes.size() / 2);
  o->n_lexicon_slots = g->lex.n_slots;
  o->byte_complete = g->vocab.byte_complete ? 1 : 0;
  o->overlay_capacity = overlay_capacity();
  return GRID_OK;
}

extern "C" int grid_add_lexicon(grid_compiled* g, const grid_lexicon_args* la, int32_t* slot) {
  clear_error();
  if (!g || !la || !slot || (la->n_categories > 0 && (!la->names || !la->words)))
    return fail(GRID_E_ARG, "null argument");
  try {
    std::vector<std::pair<std::string, std::vector<std::string>>> cats;
    for (int i = 0; i < la->n_categories; ++i) {
      if (!la->names[i] || !la->words[i]) return fail(GRID_E_ARG, "null category entry");
      std::vector<std::string> words;
      std::string cur;
      for (const char* p = la->words[i];; ++p) {
        if (*p == '\n' || *p == 0) {
          if (!cur.empty()) words.push_back(cur);
          cur.clear();
          if (*p == 0) break;
        } else {
          cur += *p;
        }
      }
      cats.push_back({la->names[i], words});
    }
    if (g->lex.n_slots >= 0xFFFF) return fail(GRID_E_CAPACITY, "too many lexicon slots");
    // add_lexicon validates every word before it appends anything, so a
    // failing call leaves the handle unchanged
    add_lexicon(g->lex, g->dfa, g->gram, g->vocab, g->term_cat, cats);
    *slot = g->lex.n_slots - 1;
    // lexicon artifacts changed: device copies must be re-bound
    g->dev[GRID_ART_LEX_FLAGS] = g->dev[GRID_ART_LEX_HASH] = g->dev[GRID_ART_LEX_SLOTS] = nullptr;
    g->dev[GRID_ART_LEX_PREFIX] = g->dev[GRID_ART_LEX_STRIDE] = g->dev[GRID_ART_LEX_TOKEN] = nullptr;
    g->dev[GRID_ART_LEX_CHILD] = g->dev[GRID_ART_LEX_TOKSUM] = nullptr;
    return GRID_OK;
  } catch (const Error& e) {
    return fail(e.code, e.what());
  } catch (const std::exception& e) {
    return fail(GRID_E_ARG, e.what());
  }
}

namespace {
template <class T>
void put(const std::vector<T>& v, const void** p, size_t* n) {
  *p = v.data();
  *n = v.size() * sizeof(T);
}
}  // namespace

extern "C" int grid_artifact(const grid_compiled* g, int32_t which, const void** p, size_t* n) {
  clear_error();
  if (!g || !p || !n) return fail(GRID_E_ARG, "null argument");
  switch (which) {
    case GRID_ART_DFA_DENSE: put(g->dfa.dense, p, n); break;
    case GRID_ART_DFA_CLASS: put(g->dfa.next, p, n); break;
    case GRID_ART_BYTE_CLASS: *p = g->dfa.byte_class; *n = 256; break;
    case GRID_ART_DFA_ACCEPT_OFF: put(g->dfa.accept_off, p, n); break;
    case GRID_ART_DFA_ACCEPT_LIST: put(g->dfa.accept_list, p, n); break;
    case GRID_ART_DFA_LIVE: put(g->dfa.live, p, n); break;
    case GRID_ART_ACTION: put(g->parser.action, p, n); break;
    case GRID_ART_GOTO: put(g->parser.go, p, n); break;
    case GRID_ART_PROD: put(g->parser.prod, p, n); break;
    case GRID_ART_TERM_INFO: put(g->term_info, p, n); break;
    case GRID_ART_SPELL_OFF: put(g->vocab.spell_off, p, n); break;
    case GRID_ART_SPELL_BYTES: put(g->vocab.spell_bytes, p, n); break;
    case GRID_ART_ALIAS_OFF: put(g->vocab.alias_off, p, n); break;
    case GRID_ART_ALIAS_IDS: put(g->vocab.alias_ids, p, n); break;
    case GRID_ART_TRIE_LEVEL_OFF: put(g->vocab.level_off, p, n); break;
    case GRID_ART_TRIE_NODES: put(g->vocab.trie_nodes, p, n); break;
    case GRID_ART_LEX_FLAGS: put(g->lex.flags, p, n); break;
    case GRID_ART_LEX_HASH: put(g->lex.hash, p, n); break;
    case GRID_ART_LEX_SLOTS: put(g->lex.slots, p, n); break;
    case GRID_ART_SPELL_REC: put(g->vocab.spell_rec, p, n); break;
    case GRID_ART_SPELL_TAIL: put(g->vocab.spell_tail, p, n); break;
    case GRID_ART_LEX_PREFIX: put(g->lex.prefix, p, n); break;
    case GRID_ART_SPELL_RANGE: put(g->vocab.sub_range, p, n); break;
    case GRID_ART_SPELL_OF_ID: put(g->vocab.spell_of_id, p, n); break;
    case GRID_ART_CLASS_MAP: put(g->classes.map, p, n); break;
    case GRID_ART_CLASS_OFF: put(g->classes.off, p, n); break;
    case GRID_ART_CLASS_REC: put(g->classes.rec, p, n); break;
    case GRID_ART_LEX_STRIDE: put(g->lex.stride, p, n); break;
    case GRID_ART_LEX_TOKEN: put(g->lex.token, p, n); break;
    case GRID_ART_ID_FIRST: put(g->vocab.id_first, p, n); break;
    case GRID_ART_PARSE_STATE: put(g->parser.pstate, p, n); break;
    case GRID_ART_PARSE_REDX: put(g->parser.predx, p, n); break;
    case GRID_ART_PARSE_SHIFT: put(g->parser.pshift, p, n); break;
    case GRID_ART_GOTO_HASH: put(g->parser.goto_hash, p, n); break;
    case GRID_ART_STATE_SYMBOL: put(g->parser.state_sym, p, n); break;
    case GRID_ART_LEX_CHILD: put(g->lex.child_bits, p, n); break;
    case GRID_ART_ID_HEAD: put(g->vocab.id_head, p, n); break;
    case GRID_ART_LEX_TOKSUM: put(g->lex.toksum, p, n); break;
    case GRID_ART_GOTO_SKIP: put(g->parser.go_skip, p, n); break;
    default: return fail(GRID_E_ARG, "unknown artifact " + std::to_string(which));
  }
  return GRID_OK;
}

extern "C" int grid_bind_device(grid_compiled* g, int32_t which, void* dev) {
  clear_error();
  if (!g || which < 0 || which >= GRID_ART_COUNT) return fail(GRID_E_ARG, "bad artifact");
  const void* hp;
  size_t n;
  int rc = grid_artifact(g, which, &hp, &n);
  if (rc) return rc;
  if (!dev && n > 0) return fail(GRID_E_ARG, "null device pointer");
  if (((uintptr_t)dev & 15) != 0) return fail(GRID_E_ARG, "device pointer not 16-byte aligned");
  g->dev[which] = dev;
  g->dev_bytes[which] = n;
  return GRID_OK;
}

extern "C" int grid_config_from_prefix(const grid_compiled* g, int32_t slot, const uint8_t* w,
                                       size_t n, grid_config* cfg, uint16_t* stack_out,
                                       uint32_t stack_cap, uint32_t* depth) {
  clear_error();
  if (!g || !cfg || !depth || (n > 0 && !w)) return fail(GRID_E_ARG, "null argument");
  if (slot < 0 || slot >= g->lex.n_slots) return fail(GRID_E_ARG, "lexicon slot out of range");
  try {
    std::vector<uint16_t> stack;
    int rc = host_config_from_prefix(g, slot, w, n, cfg, stack);
    if (rc == GRID_E_NOT_VIABLE) return fail(rc, "prefix is not a viable prefix of the language");
    if (rc) return fail(rc, "config build failed");
    *depth = (uint32_t)stack.size();
    if (stack.size() > stack_cap || (!stack_out && !stack.empty()))
      return fail(GRID_E_CAPACITY, "stack needs " + std::to_string(stack.size()) + " entries");
    std::memcpy(stack_out, stack.data(), stack.size() * sizeof(uint16_t));
    return GRID_OK;
  } catch (const std::exception& e) {
    return fail(GRID_E_ARG, e.what());
  }
}

// Rolling hash of one stack on the host, from the same definition the device
// kernels use (section 6.4).
extern "C" int grid_stack_hash_host(const grid_compiled* g, const uint16_t* states, uint32_t depth, uint64_t* out) {
  clear_error();
  if (!g || (depth > 0 && (!states || !out))) return fail(GRID_E_ARG, "grid_stack_hash_host: null pointer");
  uint64_t h = 0;
  for (uint32_t i = 0; i < depth; ++i) {
    const uint32_t sv = states[i];
    if (sv >= (uint32_t)g->parser.n_states) return fail(GRID_E_ARG, "grid_stack_hash_host: entry is no LR state");
    if (i > 0) h = node_hash(h, sv, g->parser.state_sym[sv]);
    out[i] = h;
  }
  return GRID_OK;
}
