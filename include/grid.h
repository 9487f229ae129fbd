/*
 * grid.h -- C ABI of the MI355X grammar-mask library (libgrid.so).
 *
 * The library computes the exact next-token mask of grammar-constrained
 * decoding (Definition 4, section 4.1): for a batch of parser configurations
 * (Definition 1, section 3.2: an LALR(1) stack plus the scan state of the
 * pending lexeme) it walks every vocabulary token's bytes through the lexer
 * DFA, checks each completed terminal against the incrementally advanced
 * LALR(1) parser (Proposition 3), and writes a [B, ceil(V/32)] u32 bitmask;
 * a second call fills disallowed logits with -inf (section 2, masked decoding).
 *
 * Conventions for every call:
 *  - return value: GRID_OK (0) or a negative GRID_E_* code; a message for the
 *    last failure on the calling thread is available from grid_last_error();
 *    no C++ exception crosses this boundary;
 *  - "host" pointers are CPU memory owned by the caller and only read during
 *    the call; "device" pointers are GPU memory owned by the caller (the
 *    library never allocates device memory);
 *  - asynchronous calls enqueue work on the given HIP stream (a hipStream_t
 *    passed as void*, NULL = the default stream) and return before it runs;
 *    argument errors are reported immediately and nothing is enqueued.
 *
 * Mask layout (used by grid_mask and grid_apply): token t of row b is bit
 * (t & 31) of word mask[b * W + (t >> 5)], W = ceil(V / 32); bits for t >= V
 * are 0; special tokens are 0 except the end-of-sequence id, whose bit is
 * eos_ok.
 */
#ifndef GRID_H
#define GRID_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ------------------------------------------------------------ status codes */
#define GRID_OK 0
#define GRID_E_ARG (-1)             /* bad argument (null pointer, size, range) */
#define GRID_E_GRAMMAR_SYNTAX (-2)  /* grammar text or regex does not parse */
#define GRID_E_LALR_CONFLICT (-3)   /* projected grammar is not LALR(1) */
#define GRID_E_EMPTY_LANGUAGE (-4)  /* projection left L(G) empty (section 2, L2) */
#define GRID_E_LEXICON (-5)         /* a word is not in its category's regex (W_c in R_c) */
#define GRID_E_LEXER_GAP (-6)       /* a live non-accepting DFA state follows an accepting one */
#define GRID_E_VOCAB (-7)           /* malformed vocabulary */
#define GRID_E_NOT_VIABLE (-8)      /* prefix is not in Prefix(L) */
#define GRID_E_UNBOUND (-9)         /* a device artifact was not bound */
#define GRID_E_HIP (-10)            /* a HIP launch or runtime call failed */
#define GRID_E_CAPACITY (-11)       /* a fixed capacity is exceeded (see grid_info) */

/* Row status written by grid_mask (status_dev[b]). */
#define GRID_ROW_OK 0
#define GRID_ROW_EMPTY 1            /* no token and no EOS allowed: Proposition 8 says a
                                       viable configuration never has an empty mask */
#define GRID_ROW_BAD_CONFIG 2       /* state, slot or stack out of range */
#define GRID_ROW_OVERFLOW 4         /* a per-lane parser overlay capacity was exceeded;
                                       the row's mask is not exact */
#define GRID_ROW_NOT_VIABLE 8       /* grid_accept: the token is not allowed at the
                                       configuration (the prefix would leave Prefix(L)) */
#define GRID_ROW_FINISHED 16        /* grid_accept: the end-of-sequence token was accepted */

typedef struct grid_compiled grid_compiled;

/* ------------------------------------------------------------------ compile */
typedef struct {
  const char* grammar;            /* host: grammar text (format in the design notes) */
  size_t grammar_len;
  const char* drop_labels;        /* host: comma-separated production labels the role
                                     projection removes (section 2, L2); NULL = none */
  const uint8_t* vocab_bytes;     /* host: concatenated token spellings */
  const uint64_t* vocab_offsets;  /* host: [vocab_size + 1]; token t = bytes[off[t], off[t+1]) */
  int32_t vocab_size;             /* V >= 1 */
  const int32_t* special_ids;     /* host: ids that are never allowed (except eos_id) */
  int32_t n_special;
  int32_t eos_id;                 /* -1: none; else its bit mirrors eos_ok */
} grid_compile_args;

/* Builds the host artifacts (section 6.1, offline layer): parses the grammar,
 * applies the role projection then removes useless symbols and checks that
 * the language is not empty; builds the LALR(1) ACTION/GOTO tables (reports
 * the first conflict); builds a dense 256-wide union lexer DFA over every
 * declared terminal (minimized, with byte classes, accept lists in priority
 * order and live-terminal sets) and checks it is gap-free; builds the
 * vocabulary artifacts: the distinct spellings sorted in byte order (trie DFS
 * order; "spelling order"), a levelized CSR byte trie, and the alias table
 * mapping each spelling to every id that shares it (Definition 3).  Empty spellings count as special.
 * Copies all inputs.  *out receives a handle owned by the caller
 * (grid_free).  A vocabulary that does not contain every single byte is not
 * an error; grid_info reports it (completeness precondition (a),
 * Proposition 8). */
int grid_compile(const grid_compile_args* args, grid_compiled** out);
void grid_free(grid_compiled* g);
/* Message of the last failing call on this thread ("" if none). */
const char* grid_last_error(void);

typedef struct {
  int32_t n_terminals;      /* T (declared terminals, never renumbered by projection) */
  int32_t n_nonterminals;   /* after projection and reduction */
  int32_t n_productions;
  int32_t n_lr_states;
  int32_t n_dfa_states;     /* including the dead state 0; state 1 is the start */
  int32_t n_byte_classes;
  int32_t vocab_size;       /* V */
  int32_t mask_words;       /* W = ceil(V / 32) */
  int32_t n_spellings;      /* distinct non-special spellings */
  int32_t max_spelling_len;
  int32_t n_trie_nodes;     /* levelized trie nodes (without the root) */
  int32_t n_lexicon_slots;
  int32_t byte_complete;    /* 1 if every byte 0..255 is a token spelling */
  int32_t overlay_capacity; /* per-lane parser overlay entries in grid_mask */
} grid_info_t;
int grid_info(const grid_compiled* g, grid_info_t* out);

/* Adds a schema lexicon (section 2, L3): n_categories category terminals,
 * names[i] a terminal declared with the "category" option and words[i] its
 * allow-list W_c as '\n'-separated words.  Categories not named are
 * unrestricted for rows using this slot.  Every word must be accepted by its
 * category's regex (W_c subset of R_c, checked, Proposition 8 (d)).
 * *slot receives the new slot index (slot 0 is created by grid_compile and is
 * the empty lexicon).  Adding a slot changes the lexicon artifacts: query and
 * re-bind them afterwards. */
typedef struct {
  int32_t n_categories;
  const char* const* names;
  const char* const* words;
} grid_lexicon_args;
int grid_add_lexicon(grid_compiled* g, const grid_lexicon_args* lex, int32_t* slot);

/* ---------------------------------------------------------------- artifacts */
/* Device artifacts.  The caller allocates device memory of the reported size,
 * copies the host bytes there and binds the device pointer, which must be
 * 16-byte aligned (the kernels read artifacts with 16-byte loads; GRID_E_ARG
 * otherwise); grid_mask reads only bound artifacts (GRID_E_UNBOUND otherwise).
 * The device copy stays owned by the caller and must outlive its use. */
enum {
  GRID_ART_DFA_DENSE = 0,   /* u16 [S][256] next state, 0 = dead */
  GRID_ART_DFA_CLASS,       /* u16 [S][C] next state by byte class */
  GRID_ART_BYTE_CLASS,      /* u8  [256] byte -> class */
  GRID_ART_DFA_ACCEPT_OFF,  /* u32 [S+1] offsets into ACCEPT_LIST */
  GRID_ART_DFA_ACCEPT_LIST, /* u8  accepted terminals per state, priority order */
  GRID_ART_DFA_LIVE,        /* u32 [S][8] terminals with an accept reachable */
  GRID_ART_ACTION,          /* u16 [n_lr][T+1]: 0 error, 0x4000|s shift, 0x8000|p reduce,
                               0xC000 accept; column T is end of input */
  GRID_ART_GOTO,            /* u16 [n_lr][N] */
  GRID_ART_PROD,            /* u32 [P]: lhs | len << 16 */
  GRID_ART_TERM_INFO,       /* u32 [T]: bit0 ignored, bits 8..15 category index or 0xFF */
  GRID_ART_SPELL_OFF,       /* u32 [U+1] offsets of the distinct spellings, spelling order */
  GRID_ART_SPELL_BYTES,     /* u8  spelling bytes (+32 bytes of zero padding) */
  GRID_ART_ALIAS_OFF,       /* u32 [U+1] */
  GRID_ART_ALIAS_IDS,       /* i32 token ids per spelling */
  GRID_ART_TRIE_LEVEL_OFF,  /* u32 [Lmax+2] first node of each level (level 1 first) */
  GRID_ART_TRIE_NODES,      /* u32 [n][2]: byte | parent << 8 (parent: node index + 1, 0 =
                               root), spelling index + 1 (0 = none) */
  GRID_ART_LEX_FLAGS,       /* u16 per lexicon-trie node: bit c prefix-of-category-c,
                               bit 8+c word-of-category-c */
  GRID_ART_LEX_HASH,        /* u32 [2] per entry: key = node * 256 + byte + 1 (0 empty), child */
  GRID_ART_LEX_SLOTS,       /* u32 [12] per slot: flags base, hash base, hash mask,
                               restricted-category mask, node count, prefix-table base,
                               prefix-table mask, stride-table base, stride-table mask,
                               schema fingerprint (FNV-1a of the categories and their
                               sorted words), 2 reserved */
  GRID_ART_SPELL_REC,       /* u32 [U][4] per spelling: its first 8 bytes (little-
                               endian, zero padded), first alias id | 1 << 31 when more ids
                               share the spelling, length | overflow chunk << 8 (bytes 24..
                               of a longer spelling start at SPELL_TAIL + 16 * chunk) */
  GRID_ART_PARSE_STATE,     /* u32 [n_lr][R] with TW = the smallest power of two >= (T+1)/32
                               and R = 2*TW+2 rounded up to a multiple of 4: terminals
                               that shift (or accept), terminals reduced by the state's
                               main production, that production as lhs | length << 16
                               (0xFFFFFFFF none), extra groups | their offset in
                               PARSE_REDX << 8, offset of the state's run in
                               PARSE_SHIFT, offset of its mask run (the same targets,
                               except that a shift into a unit state -- see GOTO_SKIP --
                               goes to GOTO_SKIP from the state on the unit production's
                               left side), padding */
  GRID_ART_PARSE_REDX,      /* u32 per extra reduce group: production (lhs | length << 16),
                               TW words of terminals */
  GRID_ART_GOTO_HASH,       /* GOTO_SKIP as an open-addressing table of H = 2^k slots (k >= 6,
                               load <= 2/3), u32 [H][2]: key (state << 16 | nonterminal) + 1
                               (0 empty), target; slot of a key =
                               (key * 0x9E3779B1 mod 2^32) >> (32 - k), linear probing */
  GRID_ART_SPELL_TAIL,      /* u8 [16 * chunks]: chunk u = bytes 8..23 of spelling u (zero
                               padded), then overflow chunks with bytes 24.. of spellings
                               longer than 24 bytes, each on a 16-byte boundary */
  GRID_ART_LEX_PREFIX,      /* u32 [4] per entry, per slot an open-addressing table of every
                               lexicon-trie node of depth 1..8 keyed exactly by its bytes:
                               bytes 0..3, bytes 4..7 (little-endian, zero padded),
                               length | flags << 16 (length 0 = empty), node */
  GRID_ART_SPELL_RANGE,     /* u16 per 64 consecutive spellings (a sub-tile): lowest first
                               byte | highest first byte << 8 of its spellings */
  GRID_ART_SPELL_OF_ID,     /* u32 [V]: spelling index of each token id, 0xFFFFFFFF
                               for specials and empty tokens */
  GRID_ART_CLASS_MAP,       /* u16 [S][V]: class of token id when the scan resumes in lexer
                               DFA state q (the walk's scan state, section 4.1), local to
                               q: tokens whose lexeme programs from q are equal -- the
                               number of lexeme ends maximal munch makes inside the token,
                               the DFA states of the first three ends and the state after
                               the last byte -- share a class (verdict-equivalence classes,
                               section 4.2).  Class 0: rejected by the lexer alone, special
                               or empty; class 1: judged by walking the bytes */
  GRID_ART_CLASS_OFF,       /* u32 [S+1]: first record of each state's classes */
  GRID_ART_CLASS_REC,       /* u32 [classes][4] per class: ends (0..3, 4 = more) | 8 if
                               rejected | 16 if byte 0 ends the pending lexeme | 32 for
                               class 1; state after the last byte | state of end 0 << 16;
                               state of end 1 | state of end 2 << 16; the byte indices
                               that ended lexemes 0, 1, 2 (8 bits each, 0 if missing) */
  GRID_ART_LEX_STRIDE,      /* u32 [8] per entry, per slot an open-addressing table of every
                               lexicon-trie node of depth d > 8 keyed by its ancestor at
                               depth 8 * floor((d - 1) / 8) and its 1..8 bytes below it:
                               ancestor node, bytes lo, bytes hi (little-endian, zero
                               padded), length | flags << 16 (length 0 = empty), node,
                               3 zero words */
  GRID_ART_LEX_TOKEN,       /* u32 [slots][V]: per lexicon slot and token id, for start
                               offsets o = 0 (bits 0-15) and o = 1 (bits 16-31): the
                               prefix-of-category flags of the token's bytes from o to its
                               end (low byte) and the word-of-category flags of the first
                               lexeme maximal munch cuts from o in the start state (high
                               byte; 0 when that lexeme runs to the token's end) */
  GRID_ART_ID_FIRST,        /* u8 [V]: first byte of each token id's spelling (0 for
                               specials and empty tokens) */
  GRID_ART_PARSE_SHIFT,     /* u16 per shift entry of the ACTION table: per LR state, in
                               terminal order, the target state of every terminal whose
                               PARSE_STATE shift bit is set (0 for accept); terminal t's
                               target is entry (shift bits below t) of the state's run */
  GRID_ART_STATE_SYMBOL,    /* u32 [n_lr]: the symbol on which the LR automaton enters each
                               state (terminal id, or 0x10000 | nonterminal index;
                               0xFFFFFFFF for the initial state) -- the "goto" of the
                               rolling configuration hash */
  GRID_ART_LEX_CHILD,       /* u32 [8] per lexicon-trie node (all slots, indexed like
                               LEX_FLAGS): bit b set when the node has a child on byte b */
  GRID_ART_ID_HEAD,         /* u32 [V]: the first two bytes of each token id's spelling:
                               first byte | second byte << 8 | 0x10000 when the spelling
                               has a second byte (0 for specials and empty tokens) */
  GRID_ART_LEX_TOKSUM,      /* u8 [slots][V]: which entries of LEX_TOKEN are nonzero: bit
                               2o set when the prefix flags from offset o are, bit 2o + 1
                               when the word flags from offset o are (o = 0, 1) */
  GRID_ART_GOTO_SKIP,       /* u16 [n_lr][N]: the GOTO the kernels use.  A unit state has
                               no shift and no GOTO, and on every lookahead either reduces
                               by one production X -> A with a one-symbol right side or has
                               no action; a transition into one from state b is redirected
                               to GOTO(b, X), repeatedly (the state that reduction leads to).
                               Unit states are never left on a stack after a shift, so the
                               stacks after every shift are those of GOTO; a lookahead the
                               unit state would refuse is refused later in the chain */
  GRID_ART_COUNT
};
int grid_artifact(const grid_compiled* g, int32_t which, const void** host_ptr, size_t* bytes);
int grid_bind_device(grid_compiled* g, int32_t which, void* device_ptr);

/* ----------------------------------------------------------- configurations */
/* Device form of a configuration (Definition 1), 32 bytes.  The LALR stack
 * states of the row are stack_pool[stk_off .. stk_off + stk_depth), bottom
 * first (bottom = the initial state 0); the stack is the one right after the
 * last shift.  q is the lexer DFA state after the pending lexeme r and lexnode
 * the lexicon-trie node of r in slot `slot` (0xFFFFFFFF when r is not a
 * prefix of any lexicon word).  flags bit 0: r is empty.  rem_len = |r| and
 * rem_head holds the first min(|r|, 8) bytes of r, zero padded. */
typedef struct {
  uint32_t stk_off;
  uint32_t stk_depth;
  uint32_t lexnode;
  uint16_t q;
  uint16_t slot;
  uint32_t flags;
  uint32_t rem_len;
  uint8_t rem_head[8];
} grid_config;

/* Host advance (section 6.1, per-token step 7): lexes and parses the prefix
 * w[0..n) with the same rules as the mask and fills *cfg (stk_off = 0) and
 * stack_out[0 .. *depth).  GRID_E_NOT_VIABLE if w is not a viable prefix;
 * GRID_E_CAPACITY if the stack needs more than stack_cap entries. */
int grid_config_from_prefix(const grid_compiled* g, int32_t slot, const uint8_t* w, size_t n,
                            grid_config* cfg, uint16_t* stack_out, uint32_t stack_cap,
                            uint32_t* depth);

/* --------------------------------------------------------------------- mask */
/* Device workspace bytes grid_mask needs for B rows. */
size_t grid_mask_workspace_bytes(const grid_compiled* g, int32_t B);

/* The cold exact mask of B rows (Definition 4; per-token hot path steps 1, 2,
 * 4 on a miss, and 5, section 6.1).  cfg_dev: device grid_config[B];
 * stack_pool_dev: device u16 states the configs point into; mask_dev: device
 * u32 [B][W] (fully overwritten); eos_dev: device u8 [B] (nullable);
 * status_dev: device i32 [B] GRID_ROW_* bits (nullable); workspace_dev:
 * device scratch of at least grid_mask_workspace_bytes(g, B).  All device
 * buffers are caller-owned; asynchronous on stream. */
int grid_mask(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
              const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
              int32_t* status_dev, void* workspace_dev, size_t workspace_bytes, void* stream);

/* The same work split into its launches, for callers that time or overlap
 * them: phases is a bit set of GRID_PHASE_* run in the order below on the
 * stream.  Each phase needs the earlier ones of the same rows and workspace
 * to have run before it (earlier on the stream); the mask is exact once all
 * four have run.  grid_mask equals grid_mask_phases with GRID_PHASE_ALL. */
#define GRID_PHASE_PROLOGUE 1u      /* allowed sets, EOS gate, post-shift stacks, then
                                       the verdict of every lexeme-program class of the
                                       row's lexer state */
#define GRID_PHASE_WALK 2u          /* mask_dev in token-id order from the class map;
                                       tokens whose class needs their own bytes are
                                       marked in the row's residue bitmaps (workspace) */
#define GRID_PHASE_RESIDUE 4u       /* the marked spellings: class verdict with their own
                                       lexicon flags, else the byte walk; allowed bits
                                       are OR-ed into mask_dev */
#define GRID_PHASE_FINALIZE 8u      /* tokens the residue walk handed to the slow path,
                                       then the row status when status_dev is not null */
#define GRID_PHASE_ALL 15u
int grid_mask_phases(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                     const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                     int32_t* status_dev, void* workspace_dev, size_t workspace_bytes,
                     uint32_t phases, void* stream);

/* For callers that cannot allocate (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): grid_mask without a
 * caller workspace.  Its workspace is a static device array of the library,
 * grid_mask_noalloc_max_bytes() bytes (32 MiB) on every GPU the library runs
 * on, held until the process ends; its device address is looked up once per
 * device.  The call allocates nothing; B rows need
 * grid_mask_workspace_bytes(g, B) of it, and a larger batch fails with
 * GRID_E_CAPACITY before anything is enqueued.  Every call on one GPU uses
 * the same array, and nothing is expected in it from an earlier call: calls
 * whose work overlaps on one GPU (other streams, other host threads) race
 * and must be ordered by the caller.  Outputs and errors as grid_mask. */
size_t grid_mask_noalloc_max_bytes(void);
int grid_mask_noalloc(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                      const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                      int32_t* status_dev, void* stream);

/* --------------------------------------------------------------- mask cache */
/* A configuration-keyed mask cache (section 4.3, configuration-keyed
 * caching; the per-token hot path's cache probe and write-back, section 6.1)
 * in caller-owned device memory: an open-addressing table whose entry holds
 * one whole mask row (with its EOS byte and row status), keyed by everything
 * the row's mask depends on -- the DFA state q, the pending lexeme (length,
 * first 8 bytes, lexicon node, empty flag), the lexicon slot (one key per
 * schema, so an identifier position never reads another schema's entry:
 * Proposition 6), the stack depth and the stack -- plus a fingerprint of the
 * compiled handle.  The stack enters the key as its rolling configuration
 * hash H(top) when the caller keeps one (grid_stack_hash, grid_accept_inplace;
 * read in O(1)), else as a 128-bit content hash summed over every entry.  A
 * hit reproduces the cold row bit for bit (cache-on equals cache-off) unless
 * two stacks collide in the hash.  Entries are written once and never
 * evicted; a row whose probe window (8 slots) is full stays uncached.  Calls
 * sharing a cache may run concurrently: a slot is claimed by an atomic
 * compare-and-swap, written, then published, and only published entries are
 * read. */
#define GRID_CACHE_LOOKUP 1u   /* rows whose key is published copy the cached row */
#define GRID_CACHE_INSERT 2u   /* rows that miss claim a slot and publish their row */
/* Device bytes of a cache of n_entries entries (a power of two >= 1); 0 if
 * n_entries is not one. */
size_t grid_cache_bytes(const grid_compiled* g, int32_t n_entries);
/* Empties a cache of cache_bytes (from grid_cache_bytes) with a fill kernel,
 * asynchronous on stream. */
int grid_cache_clear(const grid_compiled* g, void* cache_dev, size_t cache_bytes, void* stream);
/* grid_mask with a cache (cache_flags: GRID_CACHE_*; a null cache or flags 0
 * is exactly grid_mask).  stack_hash_dev: device u64 rolling hash of every
 * stack-pool entry (grid_stack_hash), or NULL for the content hash; a cache
 * must be used with one kind of key only.  Hit rows skip the walk. */
int grid_mask_cached(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                     const uint16_t* stack_pool_dev, const uint64_t* stack_hash_dev, uint32_t* mask_dev,
                     uint8_t* eos_dev, int32_t* status_dev, void* workspace_dev, size_t workspace_bytes,
                     void* cache_dev, size_t cache_bytes, uint32_t cache_flags, void* stream);

/* ------------------------------------------------------------ the warm path */
/* The warm per-token path (section 4.2, the split into context-independent
 * (CI) and context-dependent (CD) tokens; section 4.3, configuration-keyed
 * caching; section 6.1 steps 4-5): a cache of every row's CI words -- the
 * allowed bits of the tokens whose lexeme program from the row's scan state
 * ends no lexeme, whose verdict therefore depends only on the scan state,
 * the pending remainder, A(sigma) and the schema lexicon -- while the CD
 * tokens are judged against the live stack on every call, never cached (the
 * end-of-sequence bit is always live).  Keys, GRID_CI_* flags:
 *  - T1 (default): Definition 5's key -- the handle's fingerprint, the scan
 *    state, the lexicon slot, the pending remainder (empty flag, length,
 *    first 8 bytes, lexicon node) and A(sigma);
 *  - GRID_CI_FAMILY, the cross-family tier T2: the grammar family's
 *    fingerprint (lexer and vocabulary, the same for every role projection of
 *    one dialect) in place of the handle's, and the schema fingerprint of the
 *    slot's lexicon (GRID_ART_LEX_SLOTS word 9) in place of the slot, which
 *    scopes every entry of a lexicon-bearing producer (Remark 1); handles
 *    of one family may share a cache;
 *  - GRID_CI_GENN (with GRID_CI_FAMILY): the remainder in the genN scanner
 *    normal form (p, q, v): with this library's gap-free lexers a remainder
 *    that has accepted has p = q and v empty, so its bytes leave the key --
 *    only under the lexicon-visibility guard (no terminal the row's lexicon
 *    restricts is live or accepting in q); otherwise the raw remainder stays.
 * A hit row takes its CI words from the entry (its CI classes are neither
 * judged nor walked); a miss computes the cold mask and, with
 * GRID_CI_INSERT, claims a slot in the prologue, writes its CI tokens' bits
 * into it as the mask kernels decide them, and publishes it when the row
 * ends with status OK (other rows release their claim).  Masks are bit-identical with and without the cache.  Entries are
 * written once and never evicted; a probe window (8 slots) that is full leaves
 * the row uncached.  Concurrent calls may share a cache (claims by atomic
 * compare-and-swap, published entries only are read). */
#define GRID_CI_LOOKUP 1u
#define GRID_CI_INSERT 2u
#define GRID_CI_FAMILY 4u
#define GRID_CI_GENN 8u
/* Device bytes of a CI-words cache of n_entries entries (a power of two); 0
 * if n_entries is not one. */
size_t grid_ci_cache_bytes(const grid_compiled* g, int32_t n_entries);
/* Empties such a cache with a fill kernel, asynchronous on stream. */
int grid_ci_cache_clear(const grid_compiled* g, void* cache_dev, size_t cache_bytes, void* stream);
/* grid_mask with the CI-words cache (a null cache or no LOOKUP/INSERT flag is
 * exactly grid_mask).  Arguments otherwise as grid_mask. */
int grid_mask_warm(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                   const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev, int32_t* status_dev,
                   void* workspace_dev, size_t workspace_bytes, void* ci_cache_dev, size_t ci_cache_bytes,
                   uint32_t ci_flags, void* stream);

/* ------------------------------------------------- rolling configuration hash */
/* The rolling configuration hash of an LR stack (section 6.4, the audit
 * chain): entry 0 (the initial state, the root) hashes to 0, entry i > 0 to
 * H_i = low64(BLAKE2b-128(H_{i-1} || u32(state_i) || u32(goto_i))) with
 * BLAKE2b as published (RFC 7693), the u64 and u32 fields little-endian,
 * goto_i the state's accessing symbol (GRID_ART_STATE_SYMBOL) and low64 the
 * first 8 digest bytes read little-endian.  A push costs one hash, a pop
 * none.  grid_stack_hash writes stack_hash_dev[stk_off + i] for every entry of
 * every row's stack (device, asynchronous; O(depth) per row, once when a
 * configuration enters the device); grid_stack_hash_host does the same for one
 * stack on the host (out[0 .. depth)); GRID_E_ARG if an entry is not an LR
 * state. */
int grid_stack_hash(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                    const uint16_t* stack_pool_dev, uint64_t* stack_hash_dev, void* stream);
int grid_stack_hash_host(const grid_compiled* g, const uint16_t* states, uint32_t depth, uint64_t* out);

/* ------------------------------------------------------------------- accept */
/* Device incremental advance (section 6.1, per-token step 7): for every row b,
 * the configuration cfg_dev[b] (stack in stack_pool_dev) followed by token
 * token_dev[b].  The token's bytes are lexed and parsed with the same rules as
 * the mask (maximal munch, contextual resolution by priority, lexicon word and
 * prefix tests, Definition 2 for the new pending lexeme); the new
 * configuration goes to cfg_out_dev[b], its stack to
 * stack_out_dev[b * stack_cap ..] (cfg_out_dev[b].stk_off = b * stack_cap).
 * status_dev[b] (nullable): GRID_ROW_OK, GRID_ROW_NOT_VIABLE (token not
 * allowed), GRID_ROW_FINISHED (the end-of-sequence token, accepted: the
 * sentence is in L), GRID_ROW_BAD_CONFIG (state, slot, lexicon node, stack
 * entry or token out of range) or GRID_ROW_OVERFLOW (stack_cap too small for
 * the advanced stack).  Whatever the status, cfg_out_dev and stack_out_dev are
 * the next step's inputs: a row that is not GRID_ROW_OK keeps its
 * configuration, with its input stack copied to its own output area; a row
 * whose input stack does not fit stack_cap gets stk_depth 0 (a configuration
 * every call reports as GRID_ROW_BAD_CONFIG).  Device buffers are
 * caller-owned and must not overlap; stack_cap >= 2.  Asynchronous on stream. */
int grid_accept(const grid_compiled* g, int32_t B, const grid_config* cfg_dev, const uint16_t* stack_pool_dev,
                const int32_t* token_dev, grid_config* cfg_out_dev, uint16_t* stack_out_dev, uint32_t stack_cap,
                int32_t* status_dev, void* stream);

/* The device incremental advance on a persistent per-row stack arena
 * (section 6.2, the interned stack arena; section 6.4, the rolling hash):
 * row b's stack lives in stack_pool_dev[b * stack_cap, (b + 1) * stack_cap)
 * (cfg_dev[b].stk_off must be b * stack_cap, else GRID_ROW_BAD_CONFIG) and is
 * advanced in place by token_dev[b] with the rules of grid_accept: entries
 * below the lowest one the step rewrites are neither read back nor written
 * (each entry's parent is the entry below it), the rewritten entries are
 * written and, when stack_hash_dev (the rolling hash of every pool entry, as
 * grid_stack_hash writes it) is not NULL, their hashes are recomputed from
 * their parents' -- one hash per pushed entry, nothing per popped one.
 * cfg_dev[b] becomes the advanced configuration.  status_dev as grid_accept;
 * a row that is not GRID_ROW_OK keeps its configuration and stack untouched;
 * a stack that needs more than 8,192 entries in one step is reported as
 * GRID_ROW_OVERFLOW (grid_accept advances it).  The previous configuration of
 * an advanced row is not kept (copy the row's region first to fork it).
 * Asynchronous on stream. */
int grid_accept_inplace(const grid_compiled* g, int32_t B, grid_config* cfg_dev, uint16_t* stack_pool_dev,
                        uint64_t* stack_hash_dev, uint32_t stack_cap, const int32_t* token_dev,
                        int32_t* status_dev, void* stream);

/* ---------------------------------------------------------------- termination */
/* Termination machinery, mode 1 (section 5, Proposition 9; section 6.1 step 3),
 * host: a legal completion of the viable prefix w[0..n) on lexicon slot
 * `slot`, as vocabulary token ids in out_tokens[0 .. *out_n) -- w followed by
 * their bytes is a sentence of L, so the end-of-sequence token may follow
 * it, and every intermediate output is a viable prefix.  The pending lexeme
 * is finished by the shortest extension that a winning terminal accepts and a
 * whitespace byte ends; then a best-first search over terminal sequences on
 * the LR stack writes, per terminal, a separator and the shortest spelling
 * that wins contextual resolution there (literal text, shortest regex
 * string, or shortest word of its category in the slot's lexicon); the bytes
 * are tokenized by greedy longest match and the result is verified to be in
 * L before it is returned.  *out_n is the prefix's token-denominated reserve:
 * a decode loop with budget b tokens writes this completion and the
 * end-of-sequence token once b <= *out_n + safety.  The search is best-first
 * under a per-state estimate (the fewest terminals finishing a kernel item),
 * so the completion is short but not proven shortest.  GRID_E_NOT_VIABLE for
 * a prefix outside Prefix(L); GRID_E_CAPACITY when the completion needs more
 * than max_tokens tokens (*out_n is then its length) or none is found within
 * the search budget (60,000 expansions, 256 MiB of search nodes).  Host
 * only; safe to call from several threads on one handle, though not during
 * grid_add_lexicon on it (the writer's tables are built once, under the
 * handle's lock). */
int grid_complete(const grid_compiled* g, int32_t slot, const uint8_t* w, size_t n, int32_t max_tokens,
                  int32_t* out_tokens, int32_t* out_n);

/* Jump-forward (section 6.1 step 6), device: the B configurations
 * cfg_dev[b] (stacks at stack_pool_dev[b * stack_cap ..], the layout of
 * grid_accept_inplace) are extended by their maximal forced span, at most
 * max_len tokens long.  Step i computes the exact mask of every row; a row
 * whose mask allows exactly one token (the end-of-sequence token included,
 * when it is the only one) takes that token as span_dev[b * max_len + i] and
 * is advanced in place by it (stack_hash_dev kept as grid_accept_inplace
 * does, or NULL); any other row gets -1 there and keeps its configuration,
 * and so do the later steps of a row that stopped (after -1 or after the
 * end-of-sequence token).  span_len_dev[b] is the number of forced tokens.
 * A forced token whose advance fails (GRID_ROW_OVERFLOW: a stack beyond the
 * in-place advance's LDS area) is taken back: the row ends its span before
 * it, on the configuration it had.  On return mask_dev / eos_dev / status_dev
 * ([B, W] u32, [B] u8, [B] i32, as grid_mask writes them) hold the mask of
 * the rows' final configurations: a row with span_len < max_len there allows
 * several tokens (or is a row that grid_mask reports with a status other
 * than GRID_ROW_OK, or one whose advance failed).  workspace: device scratch
 * of at least grid_forced_span_workspace_bytes(g, B) (grid_mask's plus 4
 * bytes per row), 256-byte aligned.  max_len + 1 mask calls and max_len
 * advances are enqueued on stream, nothing is synchronized; GRID_E_ARG for
 * null pointers, B < 1, max_len < 1, stack_cap < 2 or a short workspace. */
int grid_forced_span(const grid_compiled* g, int32_t B, grid_config* cfg_dev, uint16_t* stack_pool_dev,
                     uint64_t* stack_hash_dev, uint32_t stack_cap, int32_t max_len, int32_t* span_dev,
                     int32_t* span_len_dev, uint32_t* mask_dev, uint8_t* eos_dev, int32_t* status_dev,
                     void* workspace_dev, size_t workspace_bytes, void* stream);
/* Workspace bytes grid_forced_span needs for B rows (0 for B < 1). */
size_t grid_forced_span_workspace_bytes(const grid_compiled* g, int32_t B);

/* -------------------------------------------------------------------- apply */
#define GRID_DTYPE_F32 0
#define GRID_DTYPE_BF16 1
/* In place: logits[b * row_stride + t] = -inf for every t < V whose mask bit
 * is 0 (fp32 0xFF800000, bf16 0xFF80); other entries keep their bit patterns
 * (section 2: hard -inf masking, a soundness precondition of Proposition 7).
 * With 16-byte aligned rows an aligned group of 8 logits that holds kept
 * entries is read and written back whole (kept entries rewritten with their
 * own bits), so no other writer may touch the logits during the call.
 * mask_dev: device u32 [B][ceil(V/32)]; logits_dev: device fp32 or bf16 with
 * row_stride >= V elements; 1 <= B <= 65535 (GRID_E_ARG otherwise).
 * Asynchronous on stream. */
int grid_apply(const uint32_t* mask_dev, void* logits_dev, int32_t dtype, int32_t B, int32_t V,
               int64_t row_stride, void* stream);

#ifdef __cplusplus
}
#endif
#endif
