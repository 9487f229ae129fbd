/*
 * oracle.h -- CPU oracle for the exact grammar-constrained next-token mask.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the package smoke check and
 * the benchmark's CPU-baseline leg may load this library.  The product path
 * (the HIP library) never links, loads or calls it, and the two share no code.
 *
 * What it computes is the plain definition of the mask (Definition 4, section
 * 4.1): for a current output w and a token t, bit t is 1 iff w . bytes(t) is a
 * viable prefix of the constrained language L (Definition 2, section 3.2),
 * and the end-of-sequence bit is 1 iff w is in L.  Language membership follows
 * section 2 (three grammar layers): maximal-munch lexing over the union of all
 * terminal regexes with contextual resolution (the highest-priority candidate
 * the parser can accept wins), role projection with useless-symbol removal,
 * and schema lexicons that restrict identifier categories.
 *
 * Independence: the oracle parses grammar text with its own reader, turns each
 * terminal regex into a Thompson NFA of its own, decides parser viability with
 * an Earley recognizer (not LALR tables), and keeps lexicons as plain sets.
 * Nothing here is shared with the HIP library.
 *
 * Handles are not thread-safe; one caller thread per handle.
 */
#ifndef GRID_ORACLE_H
#define GRID_ORACLE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Compile grammar text.  drop_labels: comma-separated production labels that
 * the role projection removes (NULL or "" for none).  Returns NULL on error and
 * writes a message into err. */
void* oracle_grammar_new(const char* grammar_text, const char* drop_labels,
                         char* err, int err_len);
void oracle_grammar_free(void* g);
int oracle_num_terminals(void* g);
/* Name of terminal id (declaration order, never renumbered by projection). */
const char* oracle_terminal_name(void* g, int id);

/* Schema lexicon: n categories; cat_names[i] names a category terminal and
 * words[i] is its allow-list as '\n'-separated words.  Categories the
 * lexicon does not mention are unrestricted. */
void* oracle_lexicon_new(void* g, int n, const char** cat_names, const char** words,
                         char* err, int err_len);
void oracle_lexicon_free(void* lex);

/* Vocabulary: spellings bytes[offsets[i] .. offsets[i+1]).  Special ids and
 * empty spellings are never allowed; eos_id (or -1) carries eos_ok. */
void* oracle_vocab_new(const uint8_t* bytes, const uint64_t* offsets, int V,
                       const int32_t* special_ids, int n_special, int32_t eos_id);
void oracle_vocab_free(void* voc);

/* The mask of one row.  mode 0 re-lexes and re-parses w.bytes(t) from scratch
 * for every token t; mode 1 lexes and parses w once and re-lexes only the
 * pending lexeme followed by bytes(t) (exact, since every emission inside w was
 * forced by a byte of w).  If token_ids is NULL all V tokens are computed and
 * out_words[(V+31)/32] receives the packed mask (bit t&31 of word t>>5, bits
 * >= V zero); otherwise out_bits[i] receives the bit of token_ids[i].
 * eos_ok receives w in L.  nthreads <= 0 uses all cores.  Returns 0. */
int oracle_mask(void* g, void* lex, void* voc, const uint8_t* w, size_t n, int mode,
                const int32_t* token_ids, int n_tokens, uint32_t* out_words,
                uint8_t* out_bits, int32_t* eos_ok, int nthreads);

/* w in Prefix(L), by the operational test of Definition 2. */
int oracle_viable(void* g, void* lex, const uint8_t* w, size_t n);
/* w in L. */
int oracle_member(void* g, void* lex, const uint8_t* w, size_t n);
/* Terminals the parser accepts next after the completed lexemes of w
 * (out[T] of 0/1).  Returns 1 if w's completed lexemes parse, 0 otherwise. */
int oracle_allowed(void* g, void* lex, const uint8_t* w, size_t n, uint8_t* out);

#ifdef __cplusplus
}
#endif
#endif
