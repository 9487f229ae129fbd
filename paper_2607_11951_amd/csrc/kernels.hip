// kernels.hip -- device side of the cold exact mask and the -inf apply (gfx950).
//
// grid_mask launches, on the caller's stream:
//  1. prologue (one workgroup per row; compact LR tables and the top of the
//     row's stack in LDS): thread t runs terminal t's reduce chain and shift
//     from sigma, so A(sigma) (section 3.2, allowed terminals under table
//     compression) is the set that shifted and each one's post-shift stack (an
//     overlay above the shared read-only stack) is recorded; the allowed set
//     of every post-shift stack follows by set simulation (one reduce chain
//     for a whole terminal set), and the end-of-sequence gate (section 3.2) is
//     run after each candidate winner's shift and from sigma.  Then the
//     pending lexeme's winner, the trailing-flag tables of every lexer state
//     under A(sigma) and after the winner's shift (Definition 2), and the
//     bytes that continue the pending lexeme in the schema lexicon.
//  2. verdicts (one thread per lexeme-program class of the row's lexer
//     state): tokens whose lexeme programs from that state are equal share a
//     class (the verdict-equivalence idea of section 4.2, fixed at compile
//     time per state); each class is judged once against A(sigma) and the
//     prologue's allowed sets after a first shift -- reject, allow, walk (a
//     second shift or more than three lexeme ends) or lexicon (the verdict
//     depends on the token's own lexicon flags, section 2 L3).
//  3. stream (XCD-aware, 64 ids per wave): the mask in token-id order
//     straight from the class map, one ballot per 64 ids; lexicon classes are
//     settled by a shortcut where the token's first byte or its token-flag
//     entry answers the class's first lexicon question; the rest mark their
//     spellings in the row's residue bitmaps.
//  4. residue (one 1024-thread workgroup per compute unit): marked
//     spellings in spelling order, a few per wave; lexicon spellings re-run
//     their class verdict with their own lexicon flags; the others walk their
//     bytes (section 4.1): DFA steps in LDS, a byte that kills the DFA emits
//     the pending lexeme as the highest-priority candidate that is allowed (or
//     ignored) and passes the lexicon, later shifts simulated on the lane's LDS
//     overlay; the allowed ids are OR-ed into the mask.  A lane whose stack
//     area is too small hands its spelling to the slow path.
//  5. finalize: the slow path re-walks handed-over spellings with a large
//     stack area, then the row status (Proposition 8: a viable configuration
//     has a nonempty mask); with a mask cache, the rows' masks are published.
// grid_apply is a streaming in-place -inf fill of the masked logits.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <cstdint>
#include <string>

#include "host.h"
#include "lexhash.h"
#include "rolling_hash.h"

namespace grid {
int fail(int code, const std::string& msg);
void clear_error();
}  // namespace grid

using namespace grid;

namespace {

constexpr int kBlock = 256;          // workgroup size of most kernels
constexpr int kProThreads = 512;     // prologue workgroup size (more set-simulation jobs per row)
constexpr int kStackWin = 256;       // top of the row's stack kept in LDS (prologue)
constexpr int kPostCap = 14;         // overlay states recorded per first shift
constexpr int kTmpCap = 32;          // prologue: virtual pushes of one simulation
constexpr int kGuard = 4096;         // reduce-chain step bound
constexpr int kSlowCap = 4096;       // tokens handed to the slow path per row
constexpr int kSlowThreads = 64;
constexpr int kSlowLane = 512;       // slow path per-thread stack area (workspace)
constexpr uint32_t kRowValid = 0x600D;
constexpr size_t kWsHead = 256;      // workspace head (reserved)
constexpr int kMaxRounds = 257;      // set-simulation reruns (each peels one reduce group)

// residue walk launch shape: one 1024-thread workgroup per compute unit
constexpr int kWalkThreads = 1024;
constexpr int kFastLane = 16;        // per-lane stack area in LDS (overlay at the bottom,
                                     // virtual pushes above it)
constexpr int kRowGroup = 32;        // rows resident in LDS at once (at most)
constexpr int kWalkWin = 64;         // top stack entries of each row in the walk's LDS
constexpr int kMaxItems = 1024;      // residue work items a workgroup scans at once
constexpr int kWalkChunk = 16;       // byte-walk spellings a wave takes at a time
constexpr int kLexChunk = 32;        // lexicon spellings a wave takes at a time
constexpr int kLaneSlots = 32;       // lanes of a wave with a stack area in the residue LDS
static_assert(kWalkChunk <= kLaneSlots && kLexChunk <= kLaneSlots, "chunks fit the lane stack areas");
static_assert((kLaneSlots & (kLaneSlots - 1)) == 0, "kLaneSlots is a power of two");
static_assert(kStackWin == kBlock, "one stack-window entry per prologue thread");
constexpr uint32_t kWalkLdsMax = 160 * 1024;

struct Tables {
  const uint16_t* dfa;        // [S*C]
  const uint8_t* bclass;      // [256]
  const uint32_t* acc_off;    // [S+1]
  const uint8_t* acc_list;
  const uint32_t* live;       // [S*8]
  const uint16_t* action;     // [NS*(T+1)] (shift targets)
  const uint32_t* term_info;  // [T]
  const uint32_t* pstate;     // [NS][parse_record_words(tw)]
  const uint32_t* predx;
  const uint2* ghash;         // [H]: key, target
  const uint32_t* spell_off;  // [U+1]
  const uint8_t* spell_bytes;
  const uint4* spell_rec;     // [U]: head lo, head hi, first id | multi << 31, length | chunk << 8
  const uint4* spell_tail;    // chunk u: bytes 8..23 of spelling u; overflow chunks after
  const uint32_t* alias_off;  // [U+1]
  const int32_t* alias_ids;
  const uint32_t* spell_of_id;  // [V]
  const uint16_t* lex_flags;
  const uint32_t* lex_hash;
  const uint32_t* lex_slots;
  const uint4* lex_prefix;
  const uint4* lex_stride;    // [entries][2]
  const uint32_t* lex_token;  // [slots][V] token flags at start offsets 0 and 1
  const uint32_t* id_head;    // [V] first byte | second byte << 8 | 0x10000 if it has one
  const uint8_t* lex_toksum;  // [slots][V] nonzero bytes of each token-flag entry
  const uint32_t* lex_child;  // [nodes][8] child bytes of every lexicon-trie node
  const uint16_t* cmap;       // class of each token per lexer state [S][V]
  const uint32_t* coff;       // [S+1] first class record of each state
  const uint4* crec;          // class records
  int S, C, T, N, NS, P, U, V, W, n_slots, eos_id;
  int max_classes;            // largest class count of one lexer state
  const uint16_t* pshift;      // shift targets per LR state
  const uint16_t* go;          // dense GOTO [states][N], kNoGoto none
  int tw, n_pstate, n_predx, n_pshift, n_acc, hbits;
  const uint32_t* state_sym;  // [NS] accessing symbol of each LR state (rolling hash)
  const uint64_t* stack_hash; // rolling hash of every stack entry, or null (mask cache key)
  uint8_t* cache;             // mask cache (null: off)
  uint32_t cache_mask;        // entries - 1
  uint32_t cache_flags;       // GRID_CACHE_*
  uint32_t cache_stride;      // bytes per entry
  uint32_t fp;                // fingerprint of the compiled handle
  uint8_t* ci_cache;          // context-independent-words cache (null: off)
  uint32_t ci_mask;           // entries - 1
  uint32_t ci_flags;          // GRID_CI_*
  uint32_t ci_stride;         // bytes per entry
  uint32_t family_fp;         // fingerprint of the lexer and vocabulary (the grammar family)
  uint32_t ign[8];            // the ignored terminals (term_info bit 0), one bit each
};

// ------------------------------------------------------------- mask cache
// Entry: a 64-byte key/state header, then the row's W mask words.  state 0
// empty, 1 claimed (being written), 2 published.
struct CacheEntry {
  uint32_t state, fp, q, slot, flags, rem_len, rem_lo, rem_hi, lexnode, depth;
  uint32_t h[4];  // 128-bit content hash of the stack
  uint32_t eos, status;
};
static_assert(sizeof(CacheEntry) == 64, "cache entry header is 64 bytes");
constexpr int kCacheProbes = 8;
constexpr uint64_t kRollingKeyTag = 0x524F4C4C494E4748ull;  // key words of a rolling-hash key
constexpr uint32_t kRowCached = 0xCAC4;  // RowHeader::valid of a row served from the cache

__host__ __device__ inline uint32_t cache_stride_of(int W) { return 64u + ((uint32_t)W * 4u + 15u) / 16u * 16u; }

// Context-independent-words cache entry: a 96-byte header (state word: 0
// empty, 1 claimed, 2 published; the key), then W words holding the allowed
// bits of the row's context-independent tokens -- those whose lexeme program
// from the scan state ends no lexeme, so that their verdict depends only on
// the scan state, the pending remainder, A(sigma) and the lexicon (section
// 4.2, CI / CD split; the end-of-sequence bit is never stored).
constexpr int kCiKeyWords = 17;
constexpr uint32_t kCiHeader = 96;
__host__ __device__ inline uint32_t ci_stride_of(int W) { return kCiHeader + ((uint32_t)W * 4u + 15u) / 16u * 16u; }
// A class whose tokens end no lexeme: byte 0 continues the pending lexeme and
// no later byte ends one.
__host__ __device__ inline bool ci_class(uint32_t w0) { return (w0 & (kClassEndsMask | kClassP0 | kClassWalk)) == 0u; }

// One stack entry's share of the stack hash: a 64-bit mix of (position,
// state) under a salt; the hash is the sum over the stack, so every thread
// adds its positions in any order.
__device__ inline uint64_t stack_mix(uint32_t i, uint32_t s, uint64_t salt) {
  uint64_t z = ((uint64_t)i << 32 | s) + salt;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// ---------------------------------------------------------------- workspace
// Row header, written by the prologue: everything the walk needs of a row
// besides the tables that follow it (the walk copies header, tables and
// stack window to LDS in one piece).
struct RowHeader {
  uint32_t A[8];              // allowed terminals of sigma
  uint32_t Aw[8];             // allowed terminals after shifting the winner
  uint32_t R[8];              // terminals whose category the row's lexicon restricts
  uint32_t slot[kSlotWords];  // the row's lexicon slot record (the words Slot holds; the rest 0)
  uint32_t cont[8];           // bytes b such that (pending lexeme) b prefixes a lexicon word
  uint32_t eos_ok;
  uint32_t valid;
  int32_t winner;             // pending lexeme's winner at an emission, -1 none
  uint32_t wkind;             // 0 no winner, 1 the winner is ignored, 2 it shifts
  uint32_t stk_off, stk_depth, q, lexnode;
  uint32_t rem_lo, rem_hi, rem_len;  // first 8 bytes and length of the pending lexeme
  uint32_t slow_count;
  int32_t pstat;              // status bits from the prologue
  int32_t wstat;              // status bits from the walk
  uint32_t nonempty;          // the walk allowed some token
  int32_t cache_slot;         // mask-cache entry this row publishes to, -1 none
  int32_t fstat;              // final row status (finalize)
  uint32_t cls_base, n_cls;   // the row's lexer state's class records
  uint32_t slot_id;           // the row's lexicon slot
  int32_t ci_hit;             // context-independent-words entry serving this row, -1 none
  int32_t ci_claim;           // such an entry this row publishes to, -1 none
  uint32_t pad[14];
};
static_assert(sizeof(RowHeader) == 320, "row header is 320 bytes");

struct Post {                 // stack after shifting one allowed terminal
  uint16_t k;                 // shared base entries kept
  uint8_t m;                  // overlay entries
  uint8_t ok;
  uint16_t ov[kPostCap];
};
static_assert(sizeof(Post) == 32, "post entry is 32 bytes");
static_assert(kPostCap == 14, "the walk decodes a post entry as two 16-byte halves");

struct RowLayout {
  size_t cls, win, block, post, a2, vcode, vrule, cont2, rbits, slow, slow_ov, total;
};

__host__ __device__ inline uint32_t pad16(uint32_t x) { return (x + 15u) & ~15u; }

// One row's workspace: header; trailing-flag tables under A(sigma) and after
// the winner's shift (one byte per DFA state each); the top kWalkWin states
// of the stack; [block ends here]; post-shift stacks and allowed sets of the
// allowed terminals; the class verdicts (2 bits per class of the row's lexer
// state) and lexicon shortcuts (a byte per class); for every byte b that
// continues the pending lexeme in the lexicon, the bytes that continue it
// after b (256 bits per b, rows of other b unwritten); the residue bitmaps (one
// bit per spelling the stream kernel left to the residue pass, in spelling
// order: first those the lexicon decides, then those the byte walk decides);
// the slow path's list and stack areas.
__host__ __device__ inline RowLayout row_layout(int T, int S, int U, int max_classes) {
  RowLayout L;
  size_t o = sizeof(RowHeader);
  L.cls = o;
  o += 2 * (size_t)pad16((uint32_t)S);
  L.win = o;
  o += kWalkWin * 2;
  L.block = o;
  L.post = o;
  o += (size_t)T * sizeof(Post);
  L.a2 = o;
  o += (size_t)T * 32;
  L.vcode = o;
  o += (size_t)pad16(((uint32_t)max_classes + 3u) / 4u);
  L.vrule = o;
  o += (size_t)pad16((uint32_t)max_classes);
  L.cont2 = o;
  o += 256 * 32;
  L.rbits = o;
  o += (size_t)((U + 63) / 64) * 16;
  L.slow = o;
  o += kSlowCap * 4;
  L.slow_ov = o;
  o += (size_t)kSlowThreads * kSlowLane * 2;
  L.total = (o + 255) & ~(size_t)255;
  return L;
}

__host__ __device__ inline RowLayout row_layout(const Tables& tb) { return row_layout(tb.T, tb.S, tb.U, tb.max_classes); }

// Several global -> LDS copies (each region 16-byte aligned) in one pass:
// the regions' 16-byte chunks are numbered consecutively and every thread
// issues the loads of K chunks before it stores any, so the whole staging
// costs about one memory round trip instead of one per region.  The last,
// partial chunk of a region is copied byte by byte.
#define GRID_LDS_VOID __attribute__((address_space(3))) void
struct StageRegion {
  const uint8_t* src;
  uint8_t* dst;
  uint32_t bytes;
};

template <int N, int K>
__device__ inline void stage_regions(const StageRegion (&rg)[N], int tid, int nt) {
  uint32_t total = 0;
#pragma unroll
  for (int j = 0; j < N; ++j) total += (rg[j].bytes + 15u) / 16u;
  for (uint32_t base = tid; base < total; base += (uint32_t)nt * K) {
    uint4 v[K];
    uint8_t* dst[K];
    uint32_t left[K];  // bytes of the region from this chunk on (0: no chunk)
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const uint32_t i = base + (uint32_t)(k * nt);
      // the region holding chunk i, chosen without indexing rg at run time
      const uint8_t* src = rg[0].src;
      dst[k] = rg[0].dst;
      uint32_t bytes = rg[0].bytes, first = 0, pre = 0;
#pragma unroll
      for (int t = 0; t < N; ++t) {
        if (t > 0 && i >= pre) {
          src = rg[t].src;
          dst[k] = rg[t].dst;
          bytes = rg[t].bytes;
          first = pre;
        }
        pre += (rg[t].bytes + 15u) / 16u;
      }
      const uint32_t off = (i - first) * 16u;
      left[k] = i < total ? bytes - off : 0u;
      src += off;
      dst[k] += off;
      v[k] = make_uint4(0, 0, 0, 0);
      if (left[k] >= 16u) {
        v[k] = *reinterpret_cast<const uint4*>(src);
      } else if (left[k] > 0) {
        uint32_t w[4] = {0, 0, 0, 0};
#pragma unroll
        for (int b = 0; b < 16; ++b)  // independent loads, all in flight
          if ((uint32_t)b < left[k]) w[b >> 2] |= (uint32_t)src[b] << (8 * (b & 3));
        v[k] = make_uint4(w[0], w[1], w[2], w[3]);
      }
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
      if (left[k] >= 16u) {
        *reinterpret_cast<uint4*>(dst[k]) = v[k];
      } else if (left[k] > 0) {
        const uint32_t w[4] = {v[k].x, v[k].y, v[k].z, v[k].w};
#pragma unroll
        for (int b = 0; b < 16; ++b)
          if ((uint32_t)b < left[k]) dst[k][b] = (uint8_t)(w[b >> 2] >> (8 * (b & 3)));
      }
    }
  }
}

// Global -> LDS copies by direct global-to-LDS loads (global_load_lds, 16
// bytes a lane): no registers hold the data on the way, so every load of the
// staging is issued before any is waited for and the whole staging costs
// about one memory round trip.  A region's full 16-byte chunks are cut into
// blocks of 64 (one wave instruction writes 1 KB at a wave-uniform LDS
// address, lane l at +16 l), dealt to the waves of the workgroup round-robin
// across all regions (first = the running block number); a region's last
// partial chunk is copied byte by byte by one thread.  Both ends of every
// region are 16-byte aligned.  The caller runs dma_wait() and a barrier
// before reading the copies.
__device__ inline uint32_t dma_region(const StageRegion& rg, int tid, int nt, uint32_t first) {
  const uint32_t lane = (uint32_t)tid & 63u, wave = (uint32_t)tid >> 6, nw = (uint32_t)nt >> 6;
  const uint32_t full = rg.bytes / 16u, nblk = (full + 63u) / 64u;
  for (uint32_t b = (wave + nw - first % nw) % nw; b < nblk; b += nw) {
    const uint32_t c = b * 64u + lane;
    if (c < full)
      __builtin_amdgcn_global_load_lds((const void*)(rg.src + 16u * c), (GRID_LDS_VOID*)(rg.dst + 64u * 16u * b), 16, 0,
                                       0);
  }
  const uint32_t tail = rg.bytes & 15u;
  if (tail && (uint32_t)tid == (first + nblk) % (uint32_t)nt)
    for (uint32_t i = rg.bytes - tail; i < rg.bytes; ++i) rg.dst[i] = rg.src[i];
  return first + nblk;
}

template <int N>
__device__ inline uint32_t dma_regions(const StageRegion (&rg)[N], int tid, int nt, uint32_t first = 0) {
#pragma unroll
  for (int j = 0; j < N; ++j) first = dma_region(rg[j], tid, nt, first);
  return first;
}

// Waits for this thread's outstanding loads, direct-to-LDS ones included.
__device__ inline void dma_wait() { __builtin_amdgcn_s_waitcnt(0); }

// Terminal set of every terminal (not the end of input), word w.
__device__ inline uint32_t all_word(int T, int w) {
  const int lo = w * 32;
  if (T >= lo + 32) return 0xFFFFFFFFu;
  if (T <= lo) return 0u;
  return (1u << (T - lo)) - 1u;
}

// ------------------------------------------------------- compact LR tables
// The tables and the lanes' stack areas sit in LDS in the prologue and the
// walk (L = true), where LDS-typed pointers make every access an LDS load;
// the rare slow path (L = false) reads them from global memory.
#define GRID_LDS __attribute__((address_space(3)))
template <bool L, class T>
struct MemSpace;
template <class T>
struct MemSpace<true, T> {
  typedef GRID_LDS T* ptr;
};
template <class T>
struct MemSpace<false, T> {
  typedef T* ptr;
};
template <bool L, class T>
using mptr = typename MemSpace<L, T>::ptr;
// plain vector types for 8- and 16-byte loads through typed pointers
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
template <bool L, class T>
__device__ inline mptr<L, T> in_mem(T* p) {
  return (mptr<L, T>)p;
}

template <bool L>
struct ParseTabs {
  mptr<L, const uint32_t> st;    // state records, parse_record_words(MW) words each
  mptr<L, const uint32_t> redx;  // extra reduce groups
  mptr<L, const u32x2> gh;       // GOTO (key, target) slots
  mptr<L, const uint16_t> sl;    // shift targets (runs per state)
  mptr<L, const uint16_t> gd;    // dense GOTO [states][N] when dense, else unused
  int T, hbits, N, dense;
};

struct ParseLds {  // byte offsets of the staged tables
  uint32_t st, redx, ghash, sl, gdense, total;
  int dense;  // GOTO as the dense table (else as the hash)
};

__host__ __device__ inline ParseLds parse_lds(const Tables& tb, uint32_t base, bool dense = false) {
  ParseLds L;
  uint32_t o = base;
  L.dense = dense ? 1 : 0;
  L.st = o;
  o += pad16((uint32_t)tb.n_pstate * 4);
  L.redx = o;
  o += pad16((uint32_t)tb.n_predx * 4);
  L.ghash = o;
  if (!dense) o += 8u << tb.hbits;
  L.gdense = o;
  if (dense) o += pad16((uint32_t)(tb.NS * tb.N * 2));
  L.sl = o;
  o += pad16((uint32_t)tb.n_pshift * 2);
  L.total = o - base;
  return L;
}

// The prologue's LR tables in LDS: GOTO as the dense table when it fits
// beside the prologue's own arrays, else as the hash.
constexpr uint32_t kPrologueParseMax = 92 * 1024;
__host__ __device__ inline ParseLds prologue_parse_lds(const Tables& tb) {
  const ParseLds d = parse_lds(tb, 0, true);
  return d.total <= kPrologueParseMax ? d : parse_lds(tb, 0, false);
}

// The prologue's dynamic LDS: the LR tables, then (when they fit beside
// them) the lexer's accept lists and live sets and the terminal info.
struct ProLds {
  ParseLds pl;
  uint32_t acc_off, acc_list, live, tinfo, total;
  int lexer;  // the lexer tables are staged (else read from global memory)
};
__host__ __device__ inline ProLds prologue_lds(const Tables& tb) {
  ProLds P;
  P.pl = prologue_parse_lds(tb);
  uint32_t o = P.pl.total;
  P.acc_off = o;
  o += pad16((uint32_t)(tb.S + 1) * 4u);
  P.acc_list = o;
  o += pad16((uint32_t)tb.n_acc);
  P.live = o;
  o += pad16((uint32_t)tb.S * 32u);
  P.tinfo = o;
  o += pad16((uint32_t)tb.T * 4u);
  P.lexer = o <= kPrologueParseMax ? 1 : 0;
  P.total = P.lexer ? o : P.pl.total;
  return P;
}

__device__ inline StageRegion parse_region(const Tables& tb, uint8_t* lds, const ParseLds& L, int which) {
  if (which == 0) return {(const uint8_t*)tb.pstate, lds + L.st, (uint32_t)tb.n_pstate * 4};
  if (which == 1) return {(const uint8_t*)tb.predx, lds + L.redx, (uint32_t)tb.n_predx * 4};
  if (which == 3) return {(const uint8_t*)tb.pshift, lds + L.sl, (uint32_t)tb.n_pshift * 2};
  if (L.dense) return {(const uint8_t*)tb.go, lds + L.gdense, (uint32_t)(tb.NS * tb.N * 2)};
  return {(const uint8_t*)tb.ghash, lds + L.ghash, 8u << tb.hbits};
}

// The LR tables in LDS (the caller stages them, see parse_region).
__device__ inline ParseTabs<true> lds_parse(const Tables& tb, uint8_t* lds, const ParseLds& L) {
  return {in_mem<true>((const uint32_t*)(lds + L.st)), in_mem<true>((const uint32_t*)(lds + L.redx)),
          in_mem<true>((const u32x2*)(lds + L.ghash)), in_mem<true>((const uint16_t*)(lds + L.sl)),
          in_mem<true>((const uint16_t*)(lds + L.gdense)), tb.T, tb.hbits, tb.N, L.dense};
}

__device__ inline ParseTabs<false> global_parse(const Tables& tb) {
  return {in_mem<false>(tb.pstate), in_mem<false>(tb.predx), in_mem<false>((const u32x2*)tb.ghash),
          in_mem<false>(tb.pshift), in_mem<false>(tb.go), tb.T, tb.hbits, tb.N, 1};
}

template <bool L>
struct BaseStack {  // the shared read-only stack of one row
  const uint16_t* pool;           // states [0, depth), global
  mptr<L, const uint16_t> win;    // copy of states [lo, depth), or unused with lo = depth
  uint32_t depth, lo;
  __device__ uint16_t at(uint32_t i) const { return i >= lo ? win[i - lo] : pool[i]; }
};

template <bool L>
__device__ __forceinline__ uint16_t goto_of(const ParseTabs<L>& pt, uint32_t s, uint32_t a) {
  if (pt.dense) return pt.gd[__umul24(s, (uint32_t)pt.N) + a];  // states and N below 2^24
  const uint32_t key = goto_key(s, a);
  const uint32_t mask = (1u << pt.hbits) - 1u;
  uint32_t h = goto_slot(key, pt.hbits);
  u32x2 e = pt.gh[h];
  // linear probing; the load factor (at most 2/3) keeps an empty slot
  for (uint32_t i = 0; e.x != key && e.x != 0u && i < mask; ++i) {
    h = (h + 1) & mask;
    e = pt.gh[h];
  }
  return e.x == key ? (uint16_t)e.y : kNoGoto;
}

// One state record: shift bits, main-reduce bits, main production (lhs |
// length << 16, kNoProd none), extra groups | offset << 8.
constexpr uint32_t kNoProd = 0xFFFFFFFFu;
template <int MW>
struct PRec {
  uint32_t sh[MW], rd[MW], main, extra;
};

template <bool L, int MW>
__device__ __forceinline__ PRec<MW> rec_of(const ParseTabs<L>& pt, uint32_t s) {
  constexpr int R = parse_record_words(MW);
  const mptr<L, const u32x4> p = (mptr<L, const u32x4>)(pt.st + s * (uint32_t)R);
  uint32_t w[R];
#pragma unroll
  for (int i = 0; i < R / 4; ++i) {
    const u32x4 v = p[i];
    w[4 * i] = v.x;
    w[4 * i + 1] = v.y;
    w[4 * i + 2] = v.z;
    w[4 * i + 3] = v.w;
  }
  PRec<MW> r;
#pragma unroll
  for (int k = 0; k < MW; ++k) {
    r.sh[k] = w[k];
    r.rd[k] = w[MW + k];
  }
  r.main = w[2 * MW];
  r.extra = w[2 * MW + 1];
  return r;
}

// Action of the terminal with set word w and bit `bit` in state s:
// kActShiftP (shift, or accept for the end-of-input column), kNoProd
// (error), else the production to reduce.
constexpr uint32_t kActShiftP = 0xFFFFFFFEu;
constexpr uint32_t kNoState = 0xFFFFFFFFu;
template <bool L, int MW>
__device__ __forceinline__ uint32_t action_of(const ParseTabs<L>& pt, uint32_t s, uint32_t w, uint32_t bit) {
  constexpr int R = parse_record_words(MW);
  const mptr<L, const uint32_t> rec = pt.st + s * (uint32_t)R;
  const uint32_t sh = rec[w], rd = rec[MW + w];  // both loads issued together
  const u32x2 me = *(mptr<L, const u32x2>)(rec + 2 * MW);
  const uint32_t hit = (sh | rd) & bit;
  uint32_t a = (sh & bit) ? kActShiftP : (hit ? me.x : kNoProd);
  const uint32_t nx = hit ? 0u : (me.y & 0xFFu);
  mptr<L, const uint32_t> g = pt.redx + (me.y >> 8);
  for (uint32_t e = 0; e < nx; ++e, g += MW + 1)  // the state's other reduce groups
    if (g[1 + w] & bit) {
      a = g[0];
      break;
    }
  return a;
}

template <bool L, int MW>
__device__ __forceinline__ uint32_t action_of(const ParseTabs<L>& pt, uint32_t s, int x) {
  return action_of<L, MW>(pt, s, (uint32_t)x >> 5, 1u << (x & 31));
}

// Target of the shift of terminal x in state s (x's shift bit is set): entry
// (shift bits below x) of the state's run of shift targets -- the mask run,
// where a shift into a unit state goes straight to where its reduction leads,
// or with lalr the LALR targets (stacks the device advance hands back).
template <bool L, int MW>
__device__ __forceinline__ uint16_t shift_target(const ParseTabs<L>& pt, uint32_t s, int x, bool lalr = false) {
  constexpr int R = parse_record_words(MW);
  static_assert(2 * MW + 3 < R, "the record holds both shift runs");
  const mptr<L, const uint32_t> rec = pt.st + s * (uint32_t)R;
  const uint32_t w = (uint32_t)x >> 5;
  uint32_t rank = 0, base = rec[2 * MW + (lalr ? 2 : 3)];
#pragma unroll
  for (int k = 0; k < MW; ++k) {
    const uint32_t bits = rec[k];
    if ((uint32_t)k < w) rank += (uint32_t)__popc(bits);
    if ((uint32_t)k == w) rank += (uint32_t)__popc(bits & ((1u << (x & 31)) - 1u));
  }
  return pt.sl[base + rank];
}

// Virtual stack base[0,k) ++ ov[0,m) ++ tmp[0,t) (k >= 1): its top state.
// In LDS the three places are one address space, so the address is selected
// and read once; a base entry below the LDS window is read from the pool.
template <bool L>
__device__ __forceinline__ uint16_t stack_at_top(const BaseStack<L>& bs, uint32_t k, int m,
                                                 mptr<L, const uint16_t> ov, int t,
                                                 mptr<L, const uint16_t> tmp) {
  if constexpr (L) {
    const uint32_t i = k - 1u;
    const bool deep = t == 0 && m == 0 && i < bs.lo;
    const mptr<L, const uint16_t> p = t > 0 ? tmp + (t - 1) : (m > 0 ? ov + (m - 1) : bs.win + (deep ? 0u : i - bs.lo));
    uint16_t v = *p;  // a valid LDS address in every case
    if (deep) v = bs.pool[i];
    return v;
  } else {
    if (t > 0) return tmp[t - 1];
    if (m > 0) return ov[m - 1];
    return bs.at(k - 1u);
  }
}

// Pops len entries from base[0,k) ++ ov[0,m) ++ tmp[0,t) (tmp first); false
// if that would empty the stack.
__device__ __forceinline__ bool pop_len(uint32_t len, uint32_t& k, int& m, int& t) {
  const uint32_t dt = min((uint32_t)t, len);
  const uint32_t dm = min((uint32_t)m, len - dt);
  const uint32_t dk = len - dt - dm;
  if (dk >= k) return false;
  t -= (int)dt;
  m -= (int)dm;
  k -= dk;
  return true;
}

// A chain step needs the state under the popped entries.  With one entry
// popped it is the state that was under the top (`below`, when known); with
// none, the top itself; else it is read -- only then, so a run of unit
// reductions waits for no stack read.
template <bool L>
__device__ __forceinline__ uint32_t goto_source(const BaseStack<L>& bs, uint32_t len, uint32_t s, uint32_t below,
                                                uint32_t k, int m, mptr<L, const uint16_t> ov, int t,
                                                mptr<L, const uint16_t> tmp) {
  uint32_t sb = len == 0 ? s : below;
  if (len > 1 || sb == kNoState) sb = stack_at_top<L>(bs, k, m, ov, t, tmp);
  return sb;
}

// Reduce chain of terminal x, not changing the stack (pushes go to tmp).  1
// shift, 2 accept (x is the end of input), 0 error, -1 capacity.
template <bool L, int MW>
__device__ __forceinline__ int sim1_test(const ParseTabs<L>& pt, const BaseStack<L>& bs, uint32_t k, int m,
                                         mptr<L, const uint16_t> ov, mptr<L, uint16_t> tmp, int tmpcap, int x) {
  const uint32_t w = (uint32_t)x >> 5, bit = 1u << (x & 31);
  int t = 0;
  uint32_t s = stack_at_top<L>(bs, k, m, ov, 0, tmp), below = kNoState;
  int res = -1;  // guard exhausted or capacity
  for (int guard = 0; guard < kGuard; ++guard) {
    const uint32_t a = action_of<L, MW>(pt, s, w, bit);
    if (a >= kActShiftP) {
      res = a == kActShiftP ? (x == pt.T ? 2 : 1) : 0;
      break;
    }
    const uint32_t len = a >> 16;
    if (!pop_len(len, k, m, t)) {
      res = 0;
      break;
    }
    const uint32_t sb = goto_source<L>(bs, len, s, below, k, m, ov, t, tmp);
    const uint16_t g = goto_of<L>(pt, sb, a & 0xFFFFu);
    if (g == kNoGoto || t >= tmpcap) {
      res = g == kNoGoto ? 0 : -1;
      break;
    }
    tmp[t++] = g;
    below = sb;
    s = g;
  }
  return res;
}

// Reduce chain of terminal x applied to (k, m, ov), then its shift.  1 shifted,
// 2 accept, 0 error, -1 capacity.
template <bool L, int MW>
__device__ __forceinline__ int sim1_shift(const ParseTabs<L>& pt, const BaseStack<L>& bs, uint32_t& k, int& m,
                                          mptr<L, uint16_t> ov, int cap, int x) {
  const uint32_t w = (uint32_t)x >> 5, bit = 1u << (x & 31);
  int t = 0;
  uint32_t s = stack_at_top<L>(bs, k, m, ov, 0, ov), below = kNoState;
  int res = -1;  // guard exhausted or capacity
  for (int guard = 0; guard < kGuard; ++guard) {
    const uint32_t a = action_of<L, MW>(pt, s, w, bit);
    if (a >= kActShiftP) {
      res = a == kActShiftP ? 1 : 0;
      break;
    }
    const uint32_t len = a >> 16;
    if (!pop_len(len, k, m, t)) {
      res = 0;
      break;
    }
    const uint32_t sb = goto_source<L>(bs, len, s, below, k, m, ov, 0, ov);
    const uint16_t g = goto_of<L>(pt, sb, a & 0xFFFFu);
    if (g == kNoGoto || m >= cap) {
      res = g == kNoGoto ? 0 : -1;
      break;
    }
    ov[m++] = g;
    below = sb;
    s = g;
  }
  if (res != 1) return res;
  if (x == pt.T) return 2;
  if (m >= cap) return -1;
  ov[m++] = shift_target<L, MW>(pt, s, x);
  return 1;
}

// Set simulation: acc |= the terminals of X that can be shifted next from
// base[0,k0) ++ ov[0,m0).  All of X runs one reduce chain; at each state the
// shifting terminals are accepted, those reduced by one production continue
// together, terminals of another reduce production of the same state rerun
// from the start (they follow the same chain up to that state, so every rerun
// peels off at least one group), the rest fail.  MW = words per set (the
// tables' TW).  0 ok, -1 capacity (acc is then incomplete).
template <bool L, int MW>
__device__ __forceinline__ int sim_set(const ParseTabs<L>& pt, const BaseStack<L>& bs, uint32_t k0, int m0,
                                       mptr<L, const uint16_t> ov, mptr<L, uint16_t> tmp, int tmpcap,
                                       const uint32_t (&X)[MW], uint32_t (&acc)[MW]) {
  uint32_t todo[MW];
#pragma unroll
  for (int w = 0; w < MW; ++w) todo[w] = X[w];
  const uint32_t s0 = stack_at_top<L>(bs, k0, m0, ov, 0, tmp);
  for (int round = 0; round < kMaxRounds; ++round) {
    uint32_t any = 0;
#pragma unroll
    for (int w = 0; w < MW; ++w) any |= todo[w];
    if (!any) return 0;
    uint32_t cur[MW];
#pragma unroll
    for (int w = 0; w < MW; ++w) {
      cur[w] = todo[w];
      todo[w] = 0;
    }
    uint32_t k = k0, s = s0, below = kNoState;
    int m = m0, t = 0;
    for (int guard = 0; guard < kGuard; ++guard) {
      const PRec<MW> r = rec_of<L, MW>(pt, s);
      uint32_t nxt[MW], live = 0;
#pragma unroll
      for (int w = 0; w < MW; ++w) {
        acc[w] |= cur[w] & r.sh[w];
        nxt[w] = cur[w] & r.rd[w];
        live |= nxt[w];
      }
      uint32_t chosen = live ? r.main : kNoProd;
      const uint32_t nx = r.extra & 0xFFu;
      mptr<L, const uint32_t> g = pt.redx + (r.extra >> 8);
      for (uint32_t e = 0; e < nx; ++e, g += MW + 1) {  // the state's other reduce groups
        uint32_t gl = 0, part[MW];
#pragma unroll
        for (int w = 0; w < MW; ++w) {
          part[w] = cur[w] & g[1 + w];
          gl |= part[w];
        }
        if (!gl) continue;
        if (chosen == kNoProd) {
          chosen = g[0];
#pragma unroll
          for (int w = 0; w < MW; ++w) nxt[w] = part[w];
        } else {
#pragma unroll
          for (int w = 0; w < MW; ++w) todo[w] |= part[w];
        }
      }
      if (chosen == kNoProd) break;
#pragma unroll
      for (int w = 0; w < MW; ++w) cur[w] = nxt[w];
      const uint32_t len = chosen >> 16;
      if (!pop_len(len, k, m, t)) break;
      const uint32_t sb = goto_source<L>(bs, len, s, below, k, m, ov, t, tmp);
      const uint16_t gs = goto_of<L>(pt, sb, chosen & 0xFFFFu);
      if (gs == kNoGoto) break;
      if (t >= tmpcap) return -1;
      tmp[t++] = gs;
      below = sb;
      s = gs;
    }
  }
  uint32_t any = 0;
#pragma unroll
  for (int w = 0; w < MW; ++w) any |= todo[w];
  return any ? -1 : 0;
}

// Allowed set of base[0,k) ++ ov[0,m): every terminal (not the end of input)
// that can be shifted next.
template <bool L, int MW>
__device__ __forceinline__ int allowed_set(const ParseTabs<L>& pt, const BaseStack<L>& bs, uint32_t k, int m,
                                           mptr<L, const uint16_t> ov, mptr<L, uint16_t> tmp, int tmpcap,
                                           uint32_t (&acc)[MW]) {
  uint32_t X[MW];
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    X[w] = all_word(pt.T, w);
    acc[w] = 0;
  }
  return sim_set<L, MW>(pt, bs, k, m, ov, tmp, tmpcap, X, acc);
}

// ---------------------------------------------------------- lexicon helpers
struct Slot {
  uint32_t fbase, hbase, hmask, restricted, nodes, pbase, pmask, sbase, smask;
};

__device__ inline Slot slot_of(const uint32_t* r) { return {r[0], r[1], r[2], r[3], r[4], r[5], r[6], r[7], r[8]}; }

__device__ inline Slot load_slot(const Tables& tb, int s) { return slot_of(tb.lex_slots + (size_t)s * kSlotWords); }

__device__ inline uint32_t lex_child(const Tables& tb, const Slot& sl, uint32_t node, uint32_t b) {
  if (node == kNoLex) return kNoLex;
  uint32_t key = lex_key(node, b);
  uint32_t h = lex_hash(key) & sl.hmask;
  for (uint32_t probe = 0; probe <= sl.hmask; ++probe, h = (h + 1) & sl.hmask) {
    uint2 e = reinterpret_cast<const uint2*>(tb.lex_hash)[sl.hbase + h];
    if (e.x == key) return e.y;
    if (e.x == 0) return kNoLex;
  }
  return kNoLex;
}

__device__ inline uint32_t lex_flags_of(const Tables& tb, const Slot& sl, uint32_t node) {
  return node == kNoLex ? 0u : tb.lex_flags[sl.fbase + node];
}

// Lexicon node and flags of the prefix given by its bytes (length 1..8): one
// probe in the slot's prefix table.  (0, kNoLex) if it is no word's prefix.
__device__ inline uint2 lexp_find(const Tables& tb, const Slot& sl, uint64_t bytes, uint32_t len) {
  const uint32_t lo = (uint32_t)bytes, hi = (uint32_t)(bytes >> 32);
  uint32_t h = lexp_hash(lo, hi, len) & sl.pmask;
  for (uint32_t probe = 0; probe <= sl.pmask; ++probe, h = (h + 1) & sl.pmask) {
    const uint4 e = tb.lex_prefix[sl.pbase + h];
    const uint32_t el = e.z & 0xFFFFu;
    if (el == 0) break;
    if (e.x == lo && e.y == hi && el == len) return make_uint2(e.z >> 16, e.w);
  }
  return make_uint2(0u, kNoLex);
}

// Flags and node of the lexicon-trie node below node anc (at a depth that is
// a multiple of 8) reached by len (1..8) more bytes: one probe in the slot's
// stride table.  (0, kNoLex) if no word has that prefix.
__device__ inline uint2 lexs_find(const Tables& tb, const Slot& sl, uint32_t anc, uint64_t bytes, uint32_t len) {
  const uint32_t lo = (uint32_t)bytes, hi = (uint32_t)(bytes >> 32);
  uint32_t h = lexs_hash(anc, lo, hi, len) & sl.smask;
  for (uint32_t probe = 0; probe <= sl.smask; ++probe, h = (h + 1) & sl.smask) {
    const uint4 e = tb.lex_stride[2 * (size_t)(sl.sbase + h)];
    const uint32_t el = e.w & 0xFFFFu;
    if (el == 0) break;
    if (e.x == anc && e.y == lo && e.z == hi && el == len) return make_uint2(e.w >> 16, tb.lex_stride[2 * (size_t)(sl.sbase + h) + 1].x);
  }
  return make_uint2(0u, kNoLex);
}

__device__ inline uint64_t low_bytes(uint64_t w, uint32_t n) { return n >= 8 ? w : w & ((1ull << (8 * n)) - 1ull); }

// Lexicon flags of a lexeme of len (1..24) bytes held in b0 b1 b2
// (little-endian, 8 bytes a word): at most three probes (prefix table, then
// stride table).
__device__ __forceinline__ uint32_t lex_flags_bytes(const Tables& tb, const Slot& sl, uint64_t b0, uint64_t b1,
                                                    uint64_t b2, uint32_t len) {
  if (len <= 8) return lexp_find(tb, sl, low_bytes(b0, len), len).x;
  uint32_t node = lexp_find(tb, sl, b0, 8).y;
  if (node == kNoLex) return 0u;
  if (len <= 16) return lexs_find(tb, sl, node, low_bytes(b1, len - 8), len - 8).x;
  node = lexs_find(tb, sl, node, b1, 8).y;
  if (node == kNoLex) return 0u;
  return lexs_find(tb, sl, node, low_bytes(b2, len - 16), len - 16).x;
}

// The pending lexeme as the lexicon sees it: its bytes while it has at most 8
// (bytes mode), else its lexicon-trie node (kNoLex once no word has it as a
// prefix).  Kept only when the row's lexicon restricts some category.
struct LexState {
  uint64_t w;
  uint32_t len;
  uint32_t node;
  uint32_t need;  // some restricted terminal was viable where the lexeme began
};

// Appends byte b to the pending lexeme.
__device__ inline void lex_push(const Tables& tb, const Slot& sl, LexState& lx, uint32_t b) {
  if (lx.len < 8) {
    lx.w |= (uint64_t)b << (8 * lx.len);
  } else if (lx.len == 8) {
    lx.node = lex_child(tb, sl, lexp_find(tb, sl, lx.w, 8).y, b);
  } else {
    lx.node = lex_child(tb, sl, lx.node, b);
  }
  ++lx.len;
}

__device__ inline uint32_t lex_flags_now(const Tables& tb, const Slot& sl, const LexState& lx) {
  if (lx.len == 0) return 0u;
  if (lx.len <= 8) return lexp_find(tb, sl, lx.w, lx.len).x;
  return lex_flags_of(tb, sl, lx.node);
}

__device__ inline bool bit_of(const uint32_t* s, int t) { return (s[t >> 5] >> (t & 31)) & 1u; }

// What a lane needs to judge terminals: term info, ignored set I, the row's
// restricted set R and the live-terminal sets of the lexer DFA (MW words per
// state, stride lstride).
struct TermView {
  const uint32_t* tinfo;
  const uint32_t* I;
  const uint32_t* R;
  const uint32_t* live;
  int lstride;
};

// Terminals a pending lexeme in DFA state q can still complete to that are
// allowed (acur) or ignored: bit 0 set if one of them has an unrestricted
// category, bit 1 if one has a restricted category (the lexicon decides for
// it).  Live sets only shrink as a lexeme grows, so a later byte of the same
// lexeme never gains a bit.
template <int MW>
__device__ inline uint32_t trail_flags(const TermView& tv, const uint32_t (&acur)[MW], int q) {
  uint32_t unres = 0, res = 0;
  const uint32_t* lv = tv.live + (size_t)q * tv.lstride;
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    const uint32_t bits = lv[w] & (acur[w] | tv.I[w]);
    unres |= bits & ~tv.R[w];
    res |= bits & tv.R[w];
  }
  return (unres ? 1u : 0u) | (res ? 2u : 0u);
}

// Lexicon half of Definition 2 for a lexeme whose trailing class is 2: some
// restricted terminal it can complete to has a category whose words it
// prefixes (lf = the lexeme's lexicon flags).
template <int MW>
__device__ inline bool trail_lex(const TermView& tv, const uint32_t (&acur)[MW], int q, uint32_t lf) {
  const uint32_t* lv = tv.live + (size_t)q * tv.lstride;
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    uint32_t r = lv[w] & (acur[w] | tv.I[w]) & tv.R[w];
    while (r) {
      const int t = w * 32 + __ffs(r) - 1;
      r &= r - 1;
      if ((lf >> ((tv.tinfo[t] >> 8) & 0xFFu)) & 1u) return true;
    }
  }
  return false;
}

// Definition 2 for a pending lexeme in DFA state q with lexicon flags lf.
template <int MW>
__device__ inline bool trail_ok(const TermView& tv, const uint32_t (&acur)[MW], int q, uint32_t lf) {
  const uint32_t f = trail_flags<MW>(tv, acur, q);
  return (f & 1u) || ((f & 2u) && trail_lex<MW>(tv, acur, q, lf));
}

// Pending lexeme's winner at an emission: the first accept-list entry (highest
// priority, ties to the lower id) that is ignored or allowed and passes the
// lexicon word test.  -1 if none.  lf_of() yields the lexeme's lexicon flags
// and is called at most once, only for an allowed candidate whose category is
// restricted.
template <int MW, class LexFlags>
__device__ inline int winner_of(const TermView& tv, const uint32_t* acc_off, const uint8_t* acc_list,
                                const uint32_t (&acur)[MW], int q, LexFlags lf_of) {
  uint32_t lf = 0;
  bool have_lf = false;
  for (uint32_t j = acc_off[q]; j < acc_off[q + 1]; ++j) {
    const int t = acc_list[j];
    bool ok = bit_of(tv.I, t);
#pragma unroll
    for (int w = 0; w < MW; ++w)
      if (w == (t >> 5)) ok = ok || ((acur[w] >> (t & 31)) & 1u);
    if (!ok) continue;
    if (bit_of(tv.R, t)) {
      if (!have_lf) {
        lf = lf_of();
        have_lf = true;
      }
      if (!((lf >> (8 + ((tv.tinfo[t] >> 8) & 0xFFu))) & 1u)) continue;
    }
    return t;
  }
  return -1;
}

// -------------------------------------------------- CI-words cache key
// The key of a row's context-independent words (section 4.3): per handle
// (T1, Definition 5's key) -- the handle's fingerprint, the scan state q, the
// lexicon slot, the pending remainder (empty flag, length, first 8 bytes,
// lexicon node) and A(sigma) -- or, with GRID_CI_FAMILY (the cross-family
// tier T2), the grammar family's fingerprint (lexer and vocabulary: every
// role projection of one dialect shares it, since projections never
// renumber terminals) and the slot's schema fingerprint, which scopes every
// entry of a lexicon-bearing producer (Remark 1).  With GRID_CI_GENN the T2
// remainder is taken in the genN scanner normal form: under this build's
// gap-free lexers a remainder that has accepted has its last accept at its
// end, so (p, q, v) = (q, q, empty) and the bytes drop out of the key -- only
// under the lexicon-visibility guard (no terminal the row's lexicon
// restricts is live or accepting in q); otherwise, or while the remainder
// has not accepted, the raw remainder stays in the key.
__device__ inline void ci_key(const Tables& tb, const grid_config& cfg, const Slot& sl, const uint32_t (&a_sig)[8],
                              const uint32_t* R, uint32_t (&key)[kCiKeyWords]) {
  const bool family = (tb.ci_flags & GRID_CI_FAMILY) != 0;
  const bool empty = (cfg.flags & 1u) != 0;
  bool genn = false;
  if (family && (tb.ci_flags & GRID_CI_GENN)) {
    bool guard = true;
    const uint32_t* lv = tb.live + (size_t)cfg.q * 8;
    for (int w = 0; w < 8; ++w) guard = guard && (lv[w] & R[w]) == 0u;
    const bool accepting = tb.acc_off[cfg.q + 1] > tb.acc_off[cfg.q];
    for (uint32_t j = tb.acc_off[cfg.q]; j < tb.acc_off[cfg.q + 1]; ++j) guard = guard && !bit_of(R, tb.acc_list[j]);
    genn = guard && (accepting || empty);
  }
  const uint32_t rem_lo = (uint32_t)cfg.rem_head[0] | (uint32_t)cfg.rem_head[1] << 8 |
                          (uint32_t)cfg.rem_head[2] << 16 | (uint32_t)cfg.rem_head[3] << 24;
  const uint32_t rem_hi = (uint32_t)cfg.rem_head[4] | (uint32_t)cfg.rem_head[5] << 8 |
                          (uint32_t)cfg.rem_head[6] << 16 | (uint32_t)cfg.rem_head[7] << 24;
  key[0] = family ? (genn ? 3u : 2u) : 1u;
  key[1] = family ? tb.family_fp : tb.fp;
  key[2] = cfg.q;
  key[3] = family ? tb.lex_slots[(size_t)cfg.slot * kSlotWords + 9] : (uint32_t)cfg.slot;
  key[4] = empty ? 1u : 0u;
  key[5] = genn || empty ? 0u : cfg.rem_len;
  key[6] = genn || empty ? 0u : rem_lo;
  key[7] = genn || empty ? 0u : rem_hi;
  key[8] = genn || empty ? 0u : cfg.lexnode;
#pragma unroll
  for (int k = 0; k < 8; ++k) key[9 + k] = a_sig[k];
  (void)sl;
}

// ---------------------------------------------------------------- prologue
// One workgroup per row.  Phase 1: every terminal's reduce chain and shift
// from sigma (A(sigma) is the set that shifted) and, for an allowed terminal,
// the allowed set of the stack after its shift, with the end-of-sequence gate
// run speculatively after every candidate winner's shift and from sigma; then
// the pending lexeme's winner; then the trailing-flag tables, the lexicon
// continuation bits of the pending lexeme and the row header.
template <int MW>
__global__ __launch_bounds__(kProThreads) void prologue_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                          const uint16_t* __restrict__ pool,
                                                          uint32_t* __restrict__ mask,
                                                          uint8_t* __restrict__ eos_out,
                                                          uint8_t* __restrict__ ws, size_t rbytes) {
  extern __shared__ __align__(16) uint8_t plds[];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ uint16_t win[kStackWin];
  __shared__ uint32_t A[8], I[8], R[8], Aw[8];
  __shared__ uint16_t sim_area[kProThreads][kPostCap + kTmpCap];
  __shared__ int bad, overflow, winner, eos_ok, eos_sigma, cache_hit;
  __shared__ uint8_t eos_after[256];  // end-of-sequence test after shifting each candidate winner
  __shared__ Post posts[256];          // stack after shifting each allowed terminal
  __shared__ uint32_t a2_s[256][MW];   // allowed set after shifting each allowed terminal
  __shared__ uint8_t alist[256];       // the allowed terminals in order
  __shared__ unsigned long long hacc[2];
  uint8_t* rw = ws + kWsHead + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  const RowLayout L = row_layout(tb);
  Post* post = (Post*)(rw + L.post);
  uint32_t* a2 = (uint32_t*)(rw + L.a2);
  const grid_config cfg = cfgs[row];
  const ProLds PR = prologue_lds(tb);
  const ParseLds PL = PR.pl;
  const uint32_t depth = cfg.stk_depth;
  const uint32_t lo = depth > (uint32_t)kStackWin ? depth - kStackWin : 0;
  // one round trip to memory: the LR tables (and the lexer's accept lists and
  // live sets and the terminal info) go straight to LDS while every thread
  // loads one entry of the top kStackWin stack entries
  const bool shape_ok = cfg.q < tb.S && cfg.slot < tb.n_slots && depth >= 1;  // uniform
  if (PR.lexer) {
    const StageRegion rg[8] = {parse_region(tb, plds, PL, 0),
                               parse_region(tb, plds, PL, 1),
                               parse_region(tb, plds, PL, 2),
                               parse_region(tb, plds, PL, 3),
                               {(const uint8_t*)tb.acc_off, plds + PR.acc_off, (uint32_t)(tb.S + 1) * 4u},
                               {tb.acc_list, plds + PR.acc_list, (uint32_t)tb.n_acc},
                               {(const uint8_t*)tb.live, plds + PR.live, (uint32_t)tb.S * 32u},
                               {(const uint8_t*)tb.term_info, plds + PR.tinfo, (uint32_t)tb.T * 4u}};
    dma_regions<8>(rg, tid, kProThreads);
  } else {
    const StageRegion rg[4] = {parse_region(tb, plds, PL, 0), parse_region(tb, plds, PL, 1),
                               parse_region(tb, plds, PL, 2), parse_region(tb, plds, PL, 3)};
    dma_regions<4>(rg, tid, kProThreads);
  }
  const uint32_t* acc_off = PR.lexer ? (const uint32_t*)(plds + PR.acc_off) : tb.acc_off;
  const uint8_t* acc_list = PR.lexer ? (const uint8_t*)(plds + PR.acc_list) : tb.acc_list;
  const uint32_t* live = PR.lexer ? (const uint32_t*)(plds + PR.live) : tb.live;
  const uint32_t* tinfo = PR.lexer ? (const uint32_t*)(plds + PR.tinfo) : tb.term_info;
  uint32_t s_top = 0;
  if (shape_ok && lo + (uint32_t)tid < depth) s_top = pool[cfg.stk_off + lo + tid];
  // the row's lexicon slot, its class range and this thread's terminal info,
  // in the same round trip
  const Slot sl = shape_ok ? load_slot(tb, cfg.slot) : Slot{0, 0, 0, 0, 0, 0, 0, 0, 0};
  const uint32_t cls_lo = shape_ok ? tb.coff[cfg.q] : 0u, cls_hi = shape_ok ? tb.coff[cfg.q + 1] : 0u;
  const uint32_t ti = tid < tb.T ? tb.term_info[tid] : 0u;
  const ParseTabs<true> pt = lds_parse(tb, plds, PL);
  if (tid == 0) {
    int b = shape_ok ? 0 : 1;
    if (!b && cfg.lexnode != kNoLex && cfg.lexnode >= sl.nodes) b = 1;
    bad = b;
    overflow = 0;
    winner = -1;
    eos_ok = 0;
    eos_sigma = 0;
    cache_hit = -1;
    hacc[0] = 0;
    hacc[1] = 0;
  }
  // the residue bitmaps start empty (16-byte stores): cleared during phase 1
  // by the waves below thread 256 that have no terminal, whose later work is
  // all in LDS (so nothing waits on these stores), else here
  const int z0 = ((tb.T + 63) / 64) * 64;
  uint4* const rb = (uint4*)(rw + L.rbits);
  const int n_rb = (tb.U + 63) / 64;
  if (z0 >= 256)
    for (int i = tid; i < n_rb; i += kProThreads) rb[i] = make_uint4(0, 0, 0, 0);
  dma_wait();
  __syncthreads();
  const bool sum_hash = tb.cache && !tb.stack_hash;  // the cache key needs the whole stack's content
  if (!bad) {  // every entry is an LR state; the window goes to LDS; the content hash for the cache
    uint64_t h1 = 0, h2 = 0;
    if (lo + (uint32_t)tid < depth) {
      const uint32_t i = lo + (uint32_t)tid;
      if (s_top >= (uint32_t)tb.NS) bad = 1;
      win[tid] = (uint16_t)s_top;
      if (sum_hash) {
        h1 += stack_mix(i, s_top, 0x9E3779B97F4A7C15ull);
        h2 += stack_mix(i, s_top, 0xD1B54A32D192ED03ull);
      }
    }
    for (uint32_t i = tid; i < lo; i += kProThreads) {  // entries below the window
      const uint16_t v = pool[cfg.stk_off + i];
      if (v >= tb.NS) bad = 1;
      if (sum_hash) {
        h1 += stack_mix(i, v, 0x9E3779B97F4A7C15ull);
        h2 += stack_mix(i, v, 0xD1B54A32D192ED03ull);
      }
    }
    if (sum_hash) {
      atomicAdd(&hacc[0], (unsigned long long)h1);
      atomicAdd(&hacc[1], (unsigned long long)h2);
    }
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) {
      hdr->pstat = GRID_ROW_BAD_CONFIG;
      hdr->valid = 0;
      hdr->eos_ok = 0;
      hdr->slow_count = 0;
      hdr->wstat = 0;
      hdr->nonempty = 0;
      hdr->cache_slot = -1;
      hdr->ci_hit = -1;
      hdr->ci_claim = -1;
      if (eos_out) eos_out[row] = 0;
    }
    return;
  }
  // mask cache: probe the row's key; a published entry is the row's mask, an
  // empty slot on the way is claimed for the row when inserting
  if (tb.cache && tid == 0) {
    // the stack's part of the key: its rolling hash H(top) when the caller
    // keeps one (O(1) to read), else the content sums over every entry
    uint64_t h1 = hacc[0], h2 = hacc[1];
    if (tb.stack_hash) {
      h1 = tb.stack_hash[cfg.stk_off + depth - 1];
      h2 = kRollingKeyTag;
    }
    const uint32_t key[13] = {tb.fp,
                              cfg.q,
                              cfg.slot,
                              cfg.flags & 1u,
                              cfg.rem_len,
                              (uint32_t)cfg.rem_head[0] | (uint32_t)cfg.rem_head[1] << 8 |
                                  (uint32_t)cfg.rem_head[2] << 16 | (uint32_t)cfg.rem_head[3] << 24,
                              (uint32_t)cfg.rem_head[4] | (uint32_t)cfg.rem_head[5] << 8 |
                                  (uint32_t)cfg.rem_head[6] << 16 | (uint32_t)cfg.rem_head[7] << 24,
                              cfg.lexnode,
                              depth,
                              (uint32_t)h1,
                              (uint32_t)(h1 >> 32),
                              (uint32_t)h2,
                              (uint32_t)(h2 >> 32)};
    // home slot: every key word mixed in (rows on one stack but another
    // schema or scan state start elsewhere)
    uint64_t home = h1;
    for (int k = 0; k < 9; ++k) home = stack_mix((uint32_t)k, key[k], home);
    int hit = -1, claim = -1;
    for (int pr = 0; pr < kCacheProbes; ++pr) {
      const uint32_t idx = (uint32_t)(home + (uint64_t)pr) & tb.cache_mask;
      CacheEntry* e = (CacheEntry*)(tb.cache + (size_t)idx * tb.cache_stride);
      const uint32_t st = __hip_atomic_load(&e->state, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
      if (st == 2u) {
        const uint32_t* ek = &e->fp;
        bool same = true;
        for (int k = 0; k < 13; ++k) same = same && ek[k] == key[k];
        if (same && (tb.cache_flags & GRID_CACHE_LOOKUP)) {
          hit = (int)idx;
          break;
        }
        continue;
      }
      if (st == 0u) {
        if (!(tb.cache_flags & GRID_CACHE_INSERT)) break;
        if (atomicCAS(&e->state, 0u, 1u) == 0u) {
          uint32_t* ek = &e->fp;
          for (int k = 0; k < 13; ++k) ek[k] = key[k];
          claim = (int)idx;
          break;
        }
      }
    }
    cache_hit = hit;
    hdr->cache_slot = claim;
  } else if (tid == 0) {
    hdr->cache_slot = -1;
  }
  __syncthreads();
  if (cache_hit >= 0) {  // the cached row: mask, EOS byte, status
    const CacheEntry* e = (const CacheEntry*)(tb.cache + (size_t)cache_hit * tb.cache_stride);
    const uint32_t* src = (const uint32_t*)(e + 1);
    uint32_t* dst = mask + (size_t)row * tb.W;
    for (int i = tid; i < tb.W; i += kProThreads) dst[i] = src[i];
    if (tid == 0) {
      hdr->valid = kRowCached;
      hdr->pstat = (int32_t)e->status;
      hdr->eos_ok = e->eos;
      hdr->slow_count = 0;
      hdr->wstat = 0;
      hdr->nonempty = 1;
      hdr->cache_slot = -1;
      hdr->ci_hit = -1;
      hdr->ci_claim = -1;
      if (eos_out) eos_out[row] = (uint8_t)e->eos;
    }
    return;
  }
  if (tid < 8) {
    I[tid] = tb.ign[tid];
    R[tid] = 0;
    A[tid] = 0;
    Aw[tid] = 0;
  }
  __syncthreads();
  if (tid < tb.T) {  // restricted terminals, one per thread
    const uint32_t c = (ti >> 8) & 0xFFu;
    if (c != 0xFFu && ((sl.restricted >> c) & 1u)) atomicOr(&R[tid >> 5], 1u << (tid & 31));
  }
  const BaseStack<true> bs{pool + cfg.stk_off, in_mem<true>((const uint16_t*)win), depth, lo};
  const mptr<true, uint16_t> my = in_mem<true>(&sim_area[tid][0]);
  const TermView tv{tinfo, I, R, live, 8};
  __syncthreads();

  // phase 1: terminal t's reduce chain and shift from sigma (thread t; A(sigma)
  // is the set that shifted, the stacks after the shifts go to LDS and the
  // row's workspace); a spare thread runs the end-of-sequence gate from sigma
  // itself (empty remainder, or an ignored winner); the upper waves meanwhile
  // find the bytes that continue the pending lexeme in the lexicon (thread
  // 256 + b for byte b) and, after each, the bytes that continue it further
  // (the child bitmap of that trie node)
  static_assert(kProThreads == 512, "the upper 256 threads probe one byte value each");
  const bool rem_empty = (cfg.flags & 1u) != 0;
  if (tid >= 256) {  // whole waves
    const uint32_t b = (uint32_t)tid - 256u;
    const uint32_t n1 = rem_empty ? kNoLex : lex_child(tb, sl, cfg.lexnode, b);
    const bool c = n1 != kNoLex;
    const uint64_t bal = __ballot(c);
    if ((b & 31) == 0) hdr->cont[b >> 5] = (uint32_t)(bal >> (b & 32));
    if (c) {
      const uint4* src = reinterpret_cast<const uint4*>(tb.lex_child + (size_t)(sl.fbase + n1) * 8u);
      uint4* dst = reinterpret_cast<uint4*>(rw + L.cont2 + (size_t)b * 32u);
      dst[0] = src[0];
      dst[1] = src[1];
    }
  } else if (tid < tb.T) {
    const int t = tid;
    uint32_t k = depth;
    int m = 0;
    const int r = sim1_shift<true, MW>(pt, bs, k, m, my, kPostCap, t);
    if (r < 0 || (r == 1 && k > 0xFFFF)) overflow = 1;
    if (r == 1) {
      atomicOr(&A[t >> 5], 1u << (t & 31));
      Post p;
      p.k = (uint16_t)k;
      p.m = (uint8_t)m;
      p.ok = 1;
      for (int j = 0; j < kPostCap; ++j) p.ov[j] = j < m ? (uint16_t)my[j] : (uint16_t)0;
      posts[t] = p;
      post[t] = p;
    }
  } else if (tid == 255) {  // at most 255 terminals: never a terminal's thread
    eos_sigma = sim1_test<true, MW>(pt, bs, depth, 0, my, my, kPostCap + kTmpCap, tb.T) == 2;
  }
  if (z0 < 256 && tid >= z0 && tid < 256)
    for (int i = tid - z0; i < n_rb; i += 256 - z0) rb[i] = make_uint4(0, 0, 0, 0);
  if (tid < 256) {
#pragma unroll
    for (int w = 0; w < MW; ++w) a2_s[tid][w] = 0u;
  }
  __syncthreads();
  // phase 2: the allowed set after each allowed terminal's shift, split into
  // P jobs per terminal (job j simulates the terminals x with x mod P == j, so
  // the reduce groups, each of which costs the set simulation a rerun, spread
  // over the jobs) and sized to the workgroup; then, for every candidate
  // winner of the pending lexeme, the end-of-sequence gate after its shift
  int nA = 0;
#pragma unroll
  for (int w = 0; w < MW; ++w) nA += __popc(A[w]);
  if (tid < tb.T && bit_of(A, tid)) {
    int rank = 0;  // allowed terminals below tid
#pragma unroll
    for (int w = 0; w < MW; ++w)
      if (w < (tid >> 5)) rank += __popc(A[w]);
      else if (w == (tid >> 5)) rank += __popc(A[w] & ((1u << (tid & 31)) - 1u));
    alist[rank] = (uint8_t)tid;
  }
  __syncthreads();
  // the set jobs take the first kSetThreads threads, the gates the last wave
  // (a wave runs divergent branches one after the other)
  constexpr int kSetThreads = kProThreads - 64;
  const int P = nA > 0 ? max(1, min(64, kSetThreads / nA)) : 1;
  const int n_set = nA * P;
  const bool set_lane = tid < kSetThreads;
  for (int j = set_lane ? tid : n_set + (tid - kSetThreads); j < (set_lane ? n_set : n_set + nA);
       j += set_lane ? kSetThreads : 64) {
    const int t = alist[j < n_set ? j / P : j - n_set];
    const Post& p = posts[t];
    const mptr<true, const uint16_t> ov = in_mem<true>((const uint16_t*)p.ov);
    if (j < n_set) {
      const int part = j % P;
      uint32_t X[MW], acc[MW];
#pragma unroll
      for (int w = 0; w < MW; ++w) {
        uint32_t x = 0;
        for (int b = (part - w * 32 % P + P) % P; b < 32; b += P) x |= 1u << b;
        X[w] = x & all_word(tb.T, w);
        acc[w] = 0;
      }
      if (sim_set<true, MW>(pt, bs, p.k, p.m, ov, my, kPostCap + kTmpCap, X, acc) < 0) overflow = 1;
#pragma unroll
      for (int w = 0; w < MW; ++w)
        if (acc[w]) atomicOr(&a2_s[t][w], acc[w]);
    } else if (!rem_empty) {
      bool cand = false;
      for (uint32_t q = acc_off[cfg.q]; q < acc_off[cfg.q + 1]; ++q) cand = cand || acc_list[q] == t;
      if (cand) eos_after[t] = sim1_test<true, MW>(pt, bs, p.k, p.m, ov, my, kPostCap + kTmpCap, tb.T) == 2;
    }
  }
  // the pending lexeme's winner if a byte ends it (the gate wave's first
  // thread, while the set jobs run)
  if (tid == kSetThreads && !rem_empty) {
    uint32_t a0[MW];
#pragma unroll
    for (int w = 0; w < MW; ++w) a0[w] = A[w];
    winner = winner_of<MW>(tv, acc_off, acc_list, a0, cfg.q, [&]() { return lex_flags_of(tb, sl, cfg.lexnode); });
  }
  if (tid == kProThreads - 1) {
    // context-independent words, by the gate wave's last thread while the set
    // jobs run: probe the row's key (A(sigma) is known); a published entry
    // serves the row's CI tokens, an empty slot on the way is claimed
    int ci_hit = -1, ci_claim = -1;
    if (tb.ci_cache && !overflow) {
      uint32_t a_sig[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) a_sig[k] = A[k];
      uint32_t key[kCiKeyWords];
      ci_key(tb, cfg, sl, a_sig, R, key);
      uint64_t home = 0x8F1BBCDC2C2D6A1Bull;
      for (int k = 0; k < kCiKeyWords; ++k) home = stack_mix((uint32_t)k, key[k], home);
      for (int pr = 0; pr < kCacheProbes; ++pr) {
        const uint32_t idx = (uint32_t)(home + (uint64_t)pr) & tb.ci_mask;
        uint32_t* e = (uint32_t*)(tb.ci_cache + (size_t)idx * tb.ci_stride);
        const uint32_t st = __hip_atomic_load(e, __ATOMIC_ACQUIRE, __HIP_MEMORY_SCOPE_AGENT);
        if (st == 2u) {
          bool same = true;
          for (int k = 0; k < kCiKeyWords; ++k) same = same && e[1 + k] == key[k];
          if (same && (tb.ci_flags & GRID_CI_LOOKUP)) {
            ci_hit = (int)idx;
            break;
          }
          continue;
        }
        if (st == 0u) {
          if (!(tb.ci_flags & GRID_CI_INSERT)) break;
          if (atomicCAS(e, 0u, 1u) == 0u) {
            for (int k = 0; k < kCiKeyWords; ++k) e[1 + k] = key[k];
            ci_claim = (int)idx;
            break;
          }
        }
      }
    }
    hdr->ci_hit = ci_hit;
    hdr->ci_claim = ci_claim;
  }
  __syncthreads();
  const int w = winner;
  const bool w_shifts = w >= 0 && !bit_of(I, w);
  if (tid < tb.T && bit_of(A, tid)) {
#pragma unroll
    for (int k = 0; k < MW; ++k) a2[tid * 8 + k] = a2_s[tid][k];
  }
  if (w >= 0 && tid < MW) Aw[tid] = a2_s[w][tid];
  if (tid == 0) eos_ok = (rem_empty || (w >= 0 && !w_shifts)) ? eos_sigma : (w >= 0 ? (int)eos_after[w] : 0);
  __syncthreads();
  // phase 3: the trailing-flag tables of every DFA state under A(sigma) and
  // after the winner's shift, and the top of the stack for the residue walk
  {
    uint32_t a0[MW], aw[MW];
#pragma unroll
    for (int k = 0; k < MW; ++k) {
      a0[k] = A[k];
      aw[k] = Aw[k];
    }
    uint8_t* clsA = rw + L.cls;
    uint8_t* clsW = clsA + pad16((uint32_t)tb.S);
    for (int q = tid; q < tb.S; q += kProThreads) {
      clsA[q] = (uint8_t)trail_flags<MW>(tv, a0, q);
      clsW[q] = (uint8_t)trail_flags<MW>(tv, aw, q);
    }
    uint16_t* wwin = (uint16_t*)(rw + L.win);
    const uint32_t wlo = depth > (uint32_t)kWalkWin ? depth - kWalkWin : 0u;
    if ((uint32_t)tid < depth - wlo) wwin[tid] = win[wlo + tid - lo];
  }
  __syncthreads();
  if (tid < 8) {
    hdr->A[tid] = A[tid];
    hdr->Aw[tid] = Aw[tid];
    hdr->R[tid] = R[tid];
  }
  if (tid == 0) {  // the slot's table bases and masks (its other words are not used on the device side)
    const uint32_t sw[kSlotWords] = {sl.fbase, sl.hbase, sl.hmask, sl.restricted, sl.nodes, sl.pbase,
                                     sl.pmask, sl.sbase, sl.smask, 0u,       0u,       0u};
#pragma unroll
    for (int k = 0; k < kSlotWords; ++k) hdr->slot[k] = sw[k];
  }
  if (tid == 0) {
    hdr->eos_ok = (uint32_t)eos_ok;
    if (eos_out) eos_out[row] = (uint8_t)eos_ok;
    hdr->winner = w;
    hdr->wkind = w < 0 ? 0u : (w_shifts ? 2u : 1u);
    hdr->stk_off = cfg.stk_off;
    hdr->stk_depth = depth;
    hdr->q = cfg.q;
    hdr->lexnode = cfg.lexnode;
    hdr->rem_lo = (uint32_t)cfg.rem_head[0] | (uint32_t)cfg.rem_head[1] << 8 | (uint32_t)cfg.rem_head[2] << 16 |
                  (uint32_t)cfg.rem_head[3] << 24;
    hdr->rem_hi = (uint32_t)cfg.rem_head[4] | (uint32_t)cfg.rem_head[5] << 8 | (uint32_t)cfg.rem_head[6] << 16 |
                  (uint32_t)cfg.rem_head[7] << 24;
    hdr->rem_len = rem_empty ? 0u : cfg.rem_len;
    hdr->slow_count = 0;
    hdr->wstat = 0;
    hdr->nonempty = 0;
    hdr->slot_id = cfg.slot;
    hdr->cls_base = cls_lo;
    hdr->n_cls = cls_hi - cls_lo;
    hdr->pstat = overflow ? GRID_ROW_OVERFLOW : GRID_ROW_OK;
    hdr->valid = kRowValid;
  }
}

// ------------------------------------------------------- lane machinery
// A lane's parser side.  Mode 0: the stack is sigma and acur = A(sigma).
// Mode 1: sigma plus the shift of t1, acur = that stack's allowed set (from
// the prologue).  Mode 2: a stack of its own (base[0,k) ++ overlay[0,m)) and
// the part of its allowed set that the current lexeme can still use: after
// every shift only the terminals live in the DFA state reached by the next
// lexeme's first byte are set-simulated (live sets only shrink along a
// lexeme, so every later check of that lexeme asks about a subset of them).
template <int MW>
struct Lane {
  int mode;
  int t1;
  uint32_t k;
  int m;
  uint32_t acur[MW];
  uint4 ph;  // mode 1: first 16 bytes of the row's stack after shifting t1, loaded early
};

template <bool L>
struct RowCtx {
  const Tables* tb;
  ParseTabs<L> pt;
  BaseStack<L> bs;
  Slot sl;
  TermView tv;
  const uint32_t* acc_off;  // accept-list offsets (LDS or global)
  const uint8_t* acc_list;  // accept lists (LDS or global)
  const uint32_t* a2;       // row's allowed sets after each first shift
  int a2_stride;            // words per terminal in a2
  const uint8_t* clsA;      // trailing flags per DFA state under A(sigma), or null
  const uint8_t* clsW;      // the same after shifting the winner, or null
  int winner;               // the pending lexeme's winner (-1 none)
  const Post* post;         // row's stacks after each first shift (global)
};

// Mode 2: acur = the allowed terminals of the lane's stack among those live
// in DFA state q_next (ignored ones left out: they are always viable).  1 ok,
// -1 capacity.
template <bool L, int MW>
__device__ __forceinline__ int lane_allowed(const RowCtx<L>& rc, Lane<MW>& ln, mptr<L, uint16_t> ov, int cap,
                                            int q_next) {
  uint32_t X[MW];
  const uint32_t* lv = rc.tv.live + (size_t)q_next * rc.tv.lstride;
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    X[w] = q_next == kDead ? 0u : lv[w] & ~rc.tv.I[w];
    ln.acur[w] = 0;
  }
  return sim_set<L, MW>(rc.pt, rc.bs, ln.k, ln.m, ov, ov + ln.m, cap - ln.m, X, ln.acur) < 0 ? -1 : 1;
}

// Emits the pending lexeme in DFA state q (lexicon state lx); q_next is the
// DFA state after the next lexeme's first byte.  ov is the lane's stack area
// of cap entries: the overlay occupies [0, m), virtual pushes use [m, cap).
// 1 ok, 0 reject, -1 capacity.
template <bool L, int MW>
__device__ __forceinline__ int emit(const RowCtx<L>& rc, Lane<MW>& ln, mptr<L, uint16_t> ov, int cap, int q,
                                    const LexState& lx, int q_next) {
  const int t = winner_of<MW>(rc.tv, rc.acc_off, rc.acc_list, ln.acur, q,
                              [&]() { return lex_flags_now(*rc.tb, rc.sl, lx); });
  if (t < 0) return 0;
  // an ignored winner leaves the stack unchanged; in mode 2 the next lexeme
  // still asks anew for its live terminals (the one allowed-set call below
  // serves ignored and shifted lanes of a wave together)
  const bool ignored = bit_of(rc.tv.I, t);
  if (ignored && ln.mode != 2) return 1;
  if (!ignored && ln.mode == 0) {
    ln.mode = 1;
    ln.t1 = t;
    ln.ph = reinterpret_cast<const uint4*>(rc.post)[2 * t];  // needed at the next shift
#pragma unroll
    for (int w = 0; w < MW; ++w) ln.acur[w] = rc.a2[t * rc.a2_stride + w];
    return 1;
  }
  if (!ignored && ln.mode == 1) {  // the stack after t1 (Post: k u16, m u8, ok u8, overlay u16[kPostCap])
    const uint32_t pk = ln.ph.x & 0xFFFFu, pm = (ln.ph.x >> 16) & 0xFFu, pok = ln.ph.x >> 24;
    if (!pok || pk == 0 || pk > rc.bs.depth || pm > (uint32_t)kPostCap || (int)pm > cap) return -1;
    ln.k = pk;
    ln.m = (int)pm;
    const uint32_t lo[3] = {ln.ph.y, ln.ph.z, ln.ph.w};
#pragma unroll
    for (int j = 0; j < 6; ++j)
      if (j < ln.m) ov[j] = (uint16_t)(lo[j >> 1] >> (16 * (j & 1)));
    if (ln.m > 6) {
      const uint4 h2 = reinterpret_cast<const uint4*>(rc.post)[2 * ln.t1 + 1];
      const uint32_t hi[4] = {h2.x, h2.y, h2.z, h2.w};
#pragma unroll
      for (int j = 6; j < 14; ++j)
        if (j < ln.m) ov[j] = (uint16_t)(hi[(j - 6) >> 1] >> (16 * (j & 1)));
    }
    ln.mode = 2;
  }
  if (!ignored) {
    const int r = sim1_shift<L, MW>(rc.pt, rc.bs, ln.k, ln.m, ov, cap, t);
    if (r != 1) return r < 0 ? -1 : 0;
  }
  return lane_allowed<L, MW>(rc, ln, ov, cap, q_next);
}

struct DfaView {  // lexer DFA by byte class (LDS copy or global)
  const uint16_t* next_;
  const uint8_t* cls_;
  int C;
  __device__ uint32_t cls(uint32_t b) const { return cls_[b]; }
  __device__ int next(int q, uint32_t c) const { return next_[q * C + c]; }
};

// Walks the bytes [i, n) of one spelling from lane state (ln, q, lx); f is
// the trailing flags of the last byte taken before i (1 if none).
// byte_at(i) yields byte i, called once per i in increasing order.  The lanes
// of a wave alternate between a scan phase (every lane that can takes its
// next byte: a DFA step and the trailing class, all in LDS) and an emission
// phase (lanes whose byte killed the DFA emit together), so a wave pays for
// emissions once per emission depth rather than once per byte.  Lexicon
// lookups happen only where a lexeme ends: at an emission, and at the end of
// the spelling when only restricted terminals remain (by the shrinking of live
// sets this one check covers every byte of the lexeme).  1 allowed,
// 0 rejected, -1 capacity.
template <bool L, int MW, class ByteAt>
__device__ __forceinline__ int walk_bytes(const RowCtx<L>& rc, Lane<MW>& ln, int q, LexState lx, uint32_t i,
                                          uint32_t n, ByteAt byte_at, const DfaView& step, mptr<L, uint16_t> ov,
                                          int cap, uint32_t f) {
  const Tables& tb = *rc.tb;
  const bool track = rc.sl.restricted != 0;
  // trailing flags of a state: from the row's table while the lane's allowed
  // set is that of sigma or of the winner's shift, else computed
  const uint8_t* ctab = ln.mode == 0 ? rc.clsA : (ln.mode == 1 && ln.t1 == rc.winner ? rc.clsW : nullptr);
  int status = 2;         // 2 running, else the result
  int pend = -1;          // byte class waiting for an emission
  uint32_t pend_b = 0;    // that byte
  // look-ahead, so that a byte costs one round trip to LDS: byte i and its
  // class (b0, c0), the DFA step on it from q (nx), byte i + 1 and its class
  // (b1, c1); each byte is fetched once, in increasing order, and only below n
  uint32_t b0 = i < n ? byte_at(i) : 0u;
  uint32_t b1 = i + 1 < n ? byte_at(i + 1) : 0u;
  uint32_t c0 = step.cls(b0), c1 = step.cls(b1);
  int nx = i < n ? step.next(q, c0) : kDead;
  // f: trailing flags after the last byte taken (the caller's, before any)
  for (;;) {
    for (;;) {  // scan phase
      const bool run = status == 2 && pend < 0 && i < n;
      if (!__any(run)) break;
      if (run) {
        if (nx != kDead) {
          q = nx;
          if (lx.need) lex_push(tb, rc.sl, lx, b0);
          // byte i's flags, the step on byte i + 1 and byte i + 2's class
          // depend on q or on nothing: issued together
          const uint32_t b2 = i + 2 < n ? byte_at(i + 2) : 0u;
          const uint32_t c2 = step.cls(b2);
          const int nx1 = i + 1 < n ? step.next(q, c1) : kDead;
          f = ctab ? (uint32_t)ctab[q] : trail_flags<MW>(rc.tv, ln.acur, q);
          if (f == 0) {
            status = 0;
          } else {
            ++i;
            b0 = b1;
            c0 = c1;
            nx = nx1;
            b1 = b2;
            c1 = c2;
          }
        } else {
          pend = (int)c0;
          pend_b = b0;
        }
      }
    }
    if (status == 2 && pend < 0)  // the spelling ended inside a lexeme
      status = ((f & 1u) || trail_lex<MW>(rc.tv, ln.acur, q, lex_flags_now(tb, rc.sl, lx))) ? 1 : 0;
    const bool em = status == 2 && pend >= 0;
    if (!__any(em)) break;
    if (em) {  // emission phase
      const int r = emit<L, MW>(rc, ln, ov, cap, q, lx, step.next(kStart, (uint32_t)pend));
      if (r <= 0) {
        status = r;
      } else {
        ctab = ln.mode == 0 ? rc.clsA : (ln.mode == 1 && ln.t1 == rc.winner ? rc.clsW : nullptr);
        q = step.next(kStart, (uint32_t)pend);  // byte i starts the next lexeme
        const uint32_t b2 = q != kDead && i + 2 < n ? byte_at(i + 2) : 0u;
        const uint32_t c2 = step.cls(b2);
        const int nx1 = q != kDead && i + 1 < n ? step.next(q, c1) : kDead;
        f = q == kDead ? 0u : (ctab ? (uint32_t)ctab[q] : trail_flags<MW>(rc.tv, ln.acur, q));
        lx = LexState{pend_b, 1u, kNoLex, track && (f & 2u) ? 1u : 0u};
        if (f == 0) {
          status = 0;
        } else {
          ++i;
          b0 = b1;
          c0 = c1;
          nx = nx1;
          b1 = b2;
          c1 = c2;
        }
        pend = -1;
      }
    }
  }
  return status;
}

// Bytes 1, 2, ... of one spelling, called in that order: a 64-bit window
// holds the next bytes, taken from the record (bytes 0..7), the tail chunk
// fetched with it (bytes 8..23), then one 16-byte load per overflow chunk.
struct SpellBytes {
  uint64_t win;      // next bytes, lowest first
  uint64_t lo0, hi;  // bytes 8..15; the second half of the current chunk
  const uint4* ovf;  // overflow chunk c holds bytes 24 + 16c .. 39 + 16c
  __device__ uint32_t operator()(uint32_t i) {
    if (i >= 8 && (i & 7) == 0) {
      if (i == 8) {
        win = lo0;
      } else if ((i & 15) == 0) {
        win = hi;
      } else {
        const uint4 c = ovf[(i - 24) >> 4];
        win = (uint64_t)c.x | (uint64_t)c.y << 32;
        hi = (uint64_t)c.z | (uint64_t)c.w << 32;
      }
    }
    const uint32_t b = (uint32_t)win & 0xFFu;
    win >>= 8;
    return b;
  }
};

// ----------------------------------------------------------- class verdicts
// Codes of a class for a row (2 bits per class in the row's verdict table).
// kVerdictLexicon: the verdict depends on the schema lexicon (a lexeme's
// winner or the trailing lexeme's viability), so each token of the class is
// judged again with its own lexemes' lexicon flags.
constexpr uint32_t kVerdictReject = 0, kVerdictAllow = 1, kVerdictWalk = 2, kVerdictLexicon = 3;

// Answers of a lexicon policy besides flags: the question is open (no
// answer: the class is decided by the lexicon), or the lexeme is out of
// reach of the lookup tables (the token takes the byte walk).  kLexOpen also
// marks a lexeme whose flags were not asked for yet.
constexpr uint32_t kLexOpen = 0xFFFFFFFFu, kLexOut = 0xFFFFFFFEu;

// Verdict of one lexeme-program class for a row.  The lexemes the token
// ends are judged in order against the allowed set the parser has at that
// point: A(sigma) before any shift, the prologue's allowed set after the
// first shift (a2, a2_stride words per terminal; the live sets have
// live_stride words per DFA state), unknown after a second
// one.  Each ended lexeme's winner is the first accept-list entry (priority
// order) that is ignored or allowed and, for a restricted terminal, whose
// category has the lexeme as a word (section 2, L3); the trailing lexeme
// (state after the last byte) must still complete to an allowed or ignored
// terminal, a restricted one only where the lexeme prefixes a word of its
// category (Definition 2).  An ignored unrestricted terminal live there
// accepts it under any stack.  Lexicon flags come from lex.word(i) (lexeme
// i) and lex.trail(); a lexeme after two shifts and a token with more
// recorded ends than the record holds are left to the byte walk.  With Reg,
// the row's allowed, restricted and ignored sets are first copied to
// registers (fewer dependent LDS reads, more registers).
template <int MW, class Lex, bool Reg = true>
__device__ __forceinline__ uint32_t class_verdict(const RowHeader& h, const uint32_t* I, const uint32_t* live,
                                                  int live_stride, const uint32_t* tinfo, const uint32_t* acc_off,
                                                  const uint8_t* acc_list, const uint32_t* a2, int a2_stride,
                                                  uint4 rec, Lex& lex) {
  const uint32_t w0 = rec.x;
  if (w0 & kClassReject) return kVerdictReject;
  if (w0 & kClassWalk) return kVerdictWalk;
  const uint32_t ends = w0 & kClassEndsMask;
  const uint32_t qe[kClassEnds] = {rec.y >> 16, rec.z & 0xFFFFu, rec.z >> 16};
  // the row's sets: 0 allowed A(sigma), 1 restricted R, 2 ignored I
  uint32_t Ar[MW], Rr[MW], Ir[MW];
  if constexpr (Reg) {
#pragma unroll
    for (int w = 0; w < MW; ++w) {
      Ar[w] = h.A[w];
      Rr[w] = h.R[w];
      Ir[w] = I[w];
    }
  }
  auto bit = [&](int which, int c) -> bool {
    if constexpr (!Reg) return bit_of(which == 0 ? h.A : (which == 1 ? h.R : I), c);
    const uint32_t* set = which == 0 ? Ar : (which == 1 ? Rr : Ir);
    uint32_t word = 0;
#pragma unroll
    for (int w = 0; w < MW; ++w)
      if (w == (c >> 5)) word = set[w];
    return (word >> (c & 31)) & 1u;
  };
  int sel = -1;  // allowed set now: -1 A(sigma), t >= 0 after shifting t, -2 unknown
  const uint32_t nchk = ends > (uint32_t)kClassEnds ? (uint32_t)kClassEnds : ends;
  for (uint32_t i = 0; i < nchk; ++i) {
    int t = -1;
    if (i == 0 && (w0 & kClassP0)) {  // byte 0 ends the pending lexeme: the prologue's winner
      if (h.wkind == 0) return kVerdictReject;
      if (h.wkind == 1) continue;
      t = h.winner;
    } else {
      if (sel == -2) return kVerdictWalk;
      const uint32_t q = qe[i];
      uint32_t wf = kLexOpen;  // the lexeme's lexicon flags, asked for at most once
      for (uint32_t j = acc_off[q]; j < acc_off[q + 1]; ++j) {
        const int c = acc_list[j];
        const bool ok = bit(2, c) || (sel == -1 ? bit(0, c) : bit_of(a2 + sel * a2_stride, c));
        if (!ok) continue;
        if (bit(1, c)) {
          if (wf == kLexOpen) wf = lex.word(i);
          if (wf == kLexOpen) return kVerdictLexicon;
          if (wf == kLexOut) return kVerdictWalk;
          if (!((wf >> (8 + ((tinfo[c] >> 8) & 7u))) & 1u)) continue;
        }
        t = c;
        break;
      }
      if (t < 0) return kVerdictReject;
      if (bit(2, t)) continue;
    }
    sel = sel == -1 ? t : -2;
  }
  if (ends > (uint32_t)kClassEnds) return kVerdictWalk;
  const uint32_t* lv = live + (size_t)(rec.y & 0xFFFFu) * live_stride;
  uint32_t unres = 0, res = 0, ign = 0;
  uint32_t rw[MW];  // restricted terminals that keep the trailing lexeme viable
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    const uint32_t Aw = Reg ? Ar[w] : h.A[w], Rw = Reg ? Rr[w] : h.R[w], Iw = Reg ? Ir[w] : I[w];
    const uint32_t acur = sel == -1 ? Aw : (sel >= 0 ? a2[sel * a2_stride + w] : 0u);
    const uint32_t bits = lv[w] & (acur | Iw);
    unres |= bits & ~Rw;
    rw[w] = bits & Rw;
    res |= rw[w];
    ign |= lv[w] & Iw & ~Rw;
  }
  if (ign || (sel != -2 && unres)) return kVerdictAllow;
  if (sel == -2) return kVerdictWalk;
  if (!res) return kVerdictReject;
  const uint32_t pf = lex.trail();
  if (pf == kLexOpen) return kVerdictLexicon;
  if (pf == kLexOut) return kVerdictWalk;
  uint32_t cats = 0;
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    uint32_t r = rw[w];
    while (r) {
      cats |= 1u << ((tinfo[w * 32 + __ffs(r) - 1] >> 8) & 7u);
      r &= r - 1;
    }
  }
  return (pf & cats) ? kVerdictAllow : kVerdictReject;
}

// A lexeme of the class record that starts in the start state at byte 0 or 1
// of the token: the token-flag table (GRID_ART_LEX_TOKEN) answers for it.
// Its start offset, or -1.  Lexeme 0 and a trailing lexeme after no end hold
// the pending bytes, so they qualify only when those are empty.
__device__ __forceinline__ int covered_start(uint32_t pos, uint32_t i, bool pending_empty) {
  if (i == 0) return pending_empty ? 0 : -1;
  const uint32_t o = (pos >> (8 * (i - 1))) & 0xFFu;
  return o <= 1u ? (int)o : -1;
}

// Lexicon policy that answers the class's first lexicon question with "no
// flags" and records it (kind, start offset in the token, whether the lexeme
// holds the pending bytes); it notes whether a second question is asked.
struct LexNo {
  uint32_t pos, ends;
  bool pending_empty;
  int kind;           // first question: -1 none yet, 0 trailing prefix, 1 word
  int start;          // its start offset in the token, or -1
  bool pending;       // its lexeme holds the pending bytes
  bool second;        // a second question was asked
  __device__ void first(uint32_t i, int k) {
    kind = k;
    pending = i == 0 && !pending_empty;
    start = covered_start(pos, i, pending_empty);
  }
  __device__ uint32_t word(uint32_t i) {
    if (kind >= 0) second = true;
    else first(i, 1);
    return 0u;
  }
  __device__ uint32_t trail() {
    if (kind >= 0 || ends > (uint32_t)kClassEnds) second = true;
    else first(ends, 0);
    return 0u;
  }
};

// Shortcut of a class the lexicon decides: its verdict v_no when the answer
// to its first lexicon question is "no flags", valid when that answer leads
// to no second question.  The stream kernel knows the answer is "no flags"
// when the question's lexeme starts with the pending bytes and the token's
// first byte does not continue them in the lexicon (the row's cont table) or,
// when the lexeme also holds the token's second byte, that byte does not
// continue them after the first (the row's second-byte table); or when the
// lexeme starts at token byte 0 or 1 in the start state and the token-flag
// entry has no flags there.  Encoded as 3 (the class code) | kind << 2 (0
// pending bytes, 1 trailing prefix at o, 2 word at o) | o << 4 | v_no << 5 |
// valid << 7; for kind 0, bit 4 says the lexeme holds the token's second byte
// when the token has one (a trailing lexeme, or a word ending at offset 2 or
// later).
constexpr uint32_t kNoValid = 1u << 7;
// The class's code and, for a class the lexicon decides, its shortcut, from
// one verdict run: the run under "no flags" follows the run without token
// bytes up to the first lexicon question, so a class that asks none has its
// final verdict there, and one that asks is a lexicon class whose verdict
// under "no flags" is the run's result.  Returns the code; *rule receives
// the shortcut byte of a lexicon class.
template <int MW>
__device__ __forceinline__ uint32_t class_code(const RowHeader& h, const uint32_t* I, const uint32_t* live,
                                               const uint32_t* tinfo, const uint32_t* acc_off, const uint8_t* acc_list,
                                               const uint32_t* a2, uint4 rec, uint32_t* rule) {
  LexNo ln{rec.w, rec.x & kClassEndsMask, h.rem_len == 0, -1, -1, false, false};
  const uint32_t v = class_verdict<MW>(h, I, live, 8, tinfo, acc_off, acc_list, a2, 8, rec, ln);
  if (ln.kind < 0) return v;  // no lexicon question: the class's verdict
  *rule = kVerdictLexicon;
  if (ln.second) return kVerdictLexicon;
  if (ln.pending) {
    const bool two = ln.kind == 0 || (rec.w & 0xFFu) >= 2u;
    *rule = kVerdictLexicon | (two ? 1u << 4 : 0u) | v << 5 | kNoValid;
    return kVerdictLexicon;
  }
  if (ln.start < 0) return kVerdictLexicon;
  *rule = kVerdictLexicon | (ln.kind == 0 ? 1u : 2u) << 2 | (uint32_t)ln.start << 4 | v << 5 | kNoValid;
  return kVerdictLexicon;
}

// LDS layout of the verdict kernel: live sets and the row's allowed sets
// after one shift (8 words per DFA state / terminal), terminal info, accept
// lists.
struct VerdictLds {
  uint32_t live, a2, tinfo, acc_off, acc_list, total;
};

__host__ __device__ inline VerdictLds verdict_lds(const Tables& tb) {
  VerdictLds L;
  uint32_t o = 0;
  L.live = o;
  o += (uint32_t)tb.S * 32u;
  L.a2 = o;
  o += (uint32_t)tb.T * 32u;
  L.tinfo = o;
  o += pad16((uint32_t)tb.T * 4u);
  L.acc_off = o;
  o += pad16((uint32_t)(tb.S + 1) * 4u);
  L.acc_list = o;
  o += pad16((uint32_t)tb.n_acc);
  L.total = o;
  return L;
}

// Two 16-bit masks interleaved bit by bit: bit i of a goes to bit 2i, bit i
// of b to bit 2i + 1.
__device__ inline uint32_t interleave16(uint32_t a, uint32_t b) {
  auto spread = [](uint32_t x) {
    x &= 0xFFFFu;
    x = (x | (x << 8)) & 0x00FF00FFu;
    x = (x | (x << 4)) & 0x0F0F0F0Fu;
    x = (x | (x << 2)) & 0x33333333u;
    x = (x | (x << 1)) & 0x55555555u;
    return x;
  };
  return spread(a) | spread(b) << 1;
}

// Workgroups (row, y): the verdicts of the row's classes, one class per
// thread, workgroup y taking every gridDim.y-th group of kBlock classes; each
// wave packs its 64 two-bit codes with two ballots.  A class the lexicon
// decides also gets its shortcut byte.  The row's allowed sets after one
// shift, the accept lists, the live sets and the terminal info are staged in
// LDS first (one batched pass).
template <int MW>
__global__ __launch_bounds__(kBlock) void verdict_kernel(Tables tb, uint8_t* __restrict__ ws, size_t rbytes) {
  extern __shared__ __align__(16) uint8_t vlds[];
  __shared__ RowHeader h;
  __shared__ uint32_t I_s[8];
  const int tid = threadIdx.x, lane = tid & 63;
  uint8_t* rw = ws + kWsHead + (size_t)blockIdx.x * rbytes;
  if (tid < (int)(sizeof(RowHeader) / 4)) ((uint32_t*)&h)[tid] = ((const uint32_t*)rw)[tid];
  if (tid < 8) I_s[tid] = tb.ign[tid];
  __syncthreads();
  const uint32_t n = h.n_cls;
  if (h.valid != kRowValid || blockIdx.y * (uint32_t)kBlock >= n) return;  // uniform
  const RowLayout RL = row_layout(tb);
  const VerdictLds VL = verdict_lds(tb);
  uint32_t* live_s = (uint32_t*)(vlds + VL.live);
  uint32_t* a2_s = (uint32_t*)(vlds + VL.a2);
  uint32_t* tinfo_s = (uint32_t*)(vlds + VL.tinfo);
  uint32_t* acc_off_s = (uint32_t*)(vlds + VL.acc_off);
  uint8_t* acc_list_s = vlds + VL.acc_list;
  // the first class record is fetched while the tables are staged
  uint4 rec0 = make_uint4(0, 0, 0, 0);
  if (blockIdx.y * (uint32_t)kBlock + (uint32_t)tid < n) rec0 = tb.crec[h.cls_base + blockIdx.y * kBlock + tid];
  {
    const StageRegion rg[5] = {{(const uint8_t*)tb.live, (uint8_t*)live_s, (uint32_t)tb.S * 32u},
                               {rw + RL.a2, (uint8_t*)a2_s, (uint32_t)tb.T * 32u},
                               {(const uint8_t*)tb.term_info, (uint8_t*)tinfo_s, (uint32_t)tb.T * 4u},
                               {(const uint8_t*)tb.acc_off, (uint8_t*)acc_off_s, (uint32_t)(tb.S + 1) * 4u},
                               {tb.acc_list, acc_list_s, (uint32_t)tb.n_acc}};
    dma_regions<5>(rg, tid, kBlock);
  }
  dma_wait();
  __syncthreads();
  uint32_t* vc = (uint32_t*)(rw + RL.vcode);
  uint8_t* vr = rw + RL.vrule;
  for (uint32_t c0 = blockIdx.y * kBlock; c0 < n; c0 += gridDim.y * kBlock) {  // uniform
    const uint32_t c = c0 + tid;
    uint32_t code = kVerdictReject;
    if (c < n) {
      const uint4 rec = c0 == blockIdx.y * (uint32_t)kBlock ? rec0 : tb.crec[h.cls_base + c];
      if (h.ci_hit >= 0 && ci_class(rec.x)) {  // served by the row's cached context-independent words
        code = kVerdictReject;
      } else {
        uint32_t rule = 0;
        code = class_code<MW>(h, I_s, live_s, tinfo_s, acc_off_s, acc_list_s, a2_s, rec, &rule);
        if (code == kVerdictLexicon) vr[c] = (uint8_t)rule;
      }
    }
    const uint64_t b0 = __ballot(code & 1u), b1 = __ballot(code & 2u);
    // this wave's 64 classes are words (c0 + 64 * wave) / 16 .. + 3 of the table
    if (lane < 4) {
      const uint32_t first = c0 + (uint32_t)(tid & ~63) + 16u * (uint32_t)lane;
      if (first < n) vc[first >> 4] = interleave16((uint32_t)(b0 >> (16 * lane)), (uint32_t)(b1 >> (16 * lane)));
    }

  }
}


// ------------------------------------------------------------------ stream
// The mask in token-id order straight from the class map.  Workgroup i runs
// on XCD i mod 8 and covers one row and kStreamChunks consecutive 64-id
// chunks inside that XCD's eighth of the vocabulary, so each XCD's L2 holds
// one eighth of every lexer state's class map.  A wave turns 64 ids into two
// mask words with one ballot (class verdict "allow", or the EOS id when the
// row may end).  A token whose class the lexicon decides takes the class's
// shortcut verdict when the answer to the class's first lexicon question is
// "no flags" for it (from its first byte and the row's continuation table, or
// from its token-flag entry).  Every other undecided token marks its
// spelling in the row's residue bitmap.  Rows served from the mask cache are
// skipped; rows with a bad configuration get zero words.
constexpr int kStreamWaves = kBlock / 64;
constexpr int kStreamUnroll = 4;   // chunks per wave in flight
constexpr int kStreamRounds = 1;
constexpr int kStreamChunks = kStreamWaves * kStreamUnroll * kStreamRounds;

__host__ __device__ inline int stream_slices(int V) { return ((V + 63) / 64 + 7) / 8; }
__host__ __device__ inline int stream_groups(int V) { return (stream_slices(V) + kStreamChunks - 1) / kStreamChunks; }

__global__ __launch_bounds__(kBlock) void stream_kernel(Tables tb, uint32_t* __restrict__ mask,
                                                        uint8_t* __restrict__ ws, size_t rbytes, int B) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int x = (int)(blockIdx.x & 7u);
  const int g = (int)(blockIdx.x >> 3);
  const int row = g % B, k = g / B;
  const int nch = (tb.V + 63) / 64, cps = stream_slices(tb.V);
  const int c_lo = x * cps + k * kStreamChunks;
  const int c_hi = min(min(c_lo + kStreamChunks, (x + 1) * cps), nch);
  if (c_lo >= c_hi) return;  // uniform
  uint8_t* rw = ws + kWsHead + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  const uint32_t valid = hdr->valid;
  if (valid == kRowCached) return;
  uint32_t* mrow = mask + (size_t)row * tb.W;
  if (valid != kRowValid) {  // bad configuration: an empty row
    for (int c = c_lo + wave; c < c_hi; c += kStreamWaves)
      if (lane < 2 && 2 * c + lane < tb.W) mrow[2 * c + lane] = 0u;
    return;
  }
  const RowLayout RL = row_layout(tb);
  const uint32_t q = hdr->q;
  const int eos = hdr->eos_ok ? tb.eos_id : -1;
  // a row served by cached context-independent words ORs them into its words
  const int ci = hdr->ci_hit;
  const uint32_t* ciw = ci >= 0 ? (const uint32_t*)(tb.ci_cache + (size_t)ci * tb.ci_stride + kCiHeader) : nullptr;
  // a row that claimed an entry writes its CI tokens' bits there (the residue
  // pass adds those it decides; finalize publishes the entry)
  const int claim = hdr->ci_claim;
  uint32_t* cdst = claim >= 0 ? (uint32_t*)(tb.ci_cache + (size_t)claim * tb.ci_stride + kCiHeader) : nullptr;
  const uint4* crow = tb.crec + hdr->cls_base;
  // the row's 2-bit class codes are read where the class map points (an
  // L2-resident gather: staging all of them in LDS per workgroup cost more)
  const uint32_t* vg = (const uint32_t*)(rw + RL.vcode);
  const uint16_t* cm = tb.cmap + (size_t)q * tb.V;
  const uint8_t* tsum = tb.lex_toksum + (size_t)hdr->slot_id * tb.V;
  const uint8_t* vrule = rw + RL.vrule;
  unsigned long long* rbits = (unsigned long long*)(rw + RL.rbits);
  uint32_t cont[8];
#pragma unroll
  for (int w = 0; w < 8; ++w) cont[w] = hdr->cont[w];
  bool any = false;
  constexpr int kPer = kStreamRounds * kStreamUnroll;  // chunks per wave
  // pass 1: class ids of all of this wave's chunks (loads in flight together)
  uint32_t cls[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int c = c_lo + wave + j * kStreamWaves;
    const int id = c * 64 + lane;
    cls[j] = (c < c_hi && id < tb.V) ? (uint32_t)cm[id] : 0u;
  }
  // pass 2: codes; for a class the lexicon decides, its shortcut byte, the
  // token's first two bytes and its token-flag summary; for a token the class
  // leaves undecided, its spelling (needed below if the shortcut leaves the
  // token to the residue); again all loads in flight together
  uint32_t code[kPer], sc[kPer], hd[kPer], tf[kPer], su[kPer];
  bool cib[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int c = c_lo + wave + j * kStreamWaves;
    const int id = c * 64 + lane;
    code[j] = c < c_hi ? (vg[cls[j] >> 4] >> ((cls[j] & 15u) * 2u)) & 3u : kVerdictReject;
    const bool lexq = code[j] == kVerdictLexicon && id < tb.V;
    sc[j] = lexq ? vrule[cls[j]] : 0u;
    hd[j] = lexq ? tb.id_head[id] : 0u;
    tf[j] = lexq ? tsum[id] : 0u;
    su[j] = code[j] >= kVerdictWalk && id < tb.V ? tb.spell_of_id[id] : 0xFFFFFFFFu;
    cib[j] = cdst && c < c_hi && id < tb.V ? ci_class(crow[cls[j]].x) : false;
  }
  // pass 2b: a pending-lexeme question on a lexeme that holds the token's
  // second byte, after a first byte that continues the lexeme: the second
  // byte's bit in the row's table (0 when it cannot stop the question here)
  const uint32_t* cont2 = (const uint32_t*)(rw + RL.cont2);
  uint32_t c2[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const uint32_t fb = hd[j] & 0xFFu, sb = (hd[j] >> 8) & 0xFFu;
    const bool ask = code[j] == kVerdictLexicon && (sc[j] & kNoValid) && ((sc[j] >> 2) & 3u) == 0u &&
                     ((sc[j] >> 4) & 1u) && (hd[j] & 0x10000u) && ((cont[fb >> 5] >> (fb & 31u)) & 1u);
    c2[j] = ask ? ~(cont2[fb * 8u + (sb >> 5)] >> (sb & 31u)) & 1u : 0u;
  }
  // pass 3: shortcut verdicts, mask words, residue ids
  uint32_t resu[kPer];  // this lane's residue spellings (or ~0)
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int c = c_lo + wave + j * kStreamWaves;
    const int id = c * 64 + lane;
    resu[j] = 0xFFFFFFFFu;
    if (c >= c_hi) continue;  // uniform across the wave
    uint32_t cd = code[j];
    if (cd == kVerdictLexicon && (sc[j] & kNoValid)) {
      const uint32_t kind = (sc[j] >> 2) & 3u, fb = hd[j] & 0xFFu;
      const bool no = kind == 0 ? !((cont[fb >> 5] >> (fb & 31u)) & 1u) || c2[j] != 0u
                                : ((tf[j] >> (2 * ((sc[j] >> 4) & 1u) + (kind == 2 ? 1u : 0u))) & 1u) == 0u;
      if (no) cd = (sc[j] >> 5) & 3u;
    }
    const uint64_t al = __ballot(cd == kVerdictAllow || id == eos);
    uint64_t cw = 0;
    if (ciw) cw = (uint64_t)ciw[2 * c] | (2 * c + 1 < tb.W ? (uint64_t)ciw[2 * c + 1] << 32 : 0ull);
    any = any || (al | cw) != 0;
    if (lane < 2 && 2 * c + lane < tb.W) mrow[2 * c + lane] = (uint32_t)((al | cw) >> (32 * lane));
    if (cdst) {  // uniform: the claimed entry's words (the end-of-sequence bit is never cached)
      const uint64_t cb = __ballot(cib[j] && cd == kVerdictAllow && id < tb.V && id != tb.eos_id);
      if (lane < 2 && 2 * c + lane < tb.W) cdst[2 * c + lane] = (uint32_t)(cb >> (32 * lane));
    }
    if (cd >= kVerdictWalk && id < tb.V) resu[j] = su[j];
    code[j] = cd;
  }
  // mark the residue spellings in the row's bitmaps (lexicon or byte walk),
  // last, so no load above waits behind these atomics
  const uint32_t nsub = ((uint32_t)tb.U + 63u) / 64u;
#pragma unroll
  for (int k2 = 0; k2 < kPer; ++k2)
    if (resu[k2] != 0xFFFFFFFFu) {
      const uint32_t u = resu[k2];
      atomicOr(rbits + (code[k2] == kVerdictWalk ? nsub : 0u) + (u >> 6), 1ull << (u & 63u));
    }
  if (lane == 0 && any) hdr->nonempty = 1u;
}

// ----------------------------------------------------------------- residue
// The next value of an LDS counter for the whole wave (one atomic).
__device__ inline int wave_grab(int* ctr) {
  int v = 0;
  if ((threadIdx.x & 63) == 0) v = atomicAdd(ctr, 1);
  return __builtin_amdgcn_readfirstlane(v);
}

struct ResLds {  // byte offsets into dynamic LDS
  uint32_t dfa, bcls, tinfo, I, acc_off, acc_list, parse, live, lanes, umask, upre, rows, total;
  uint32_t block;  // bytes per resident row: header, trailing-flag tables, stack window
  int group;       // rows per group
  ParseLds pl;
};

__host__ __device__ inline ResLds res_lds_with(const Tables& tb, int mw, int B, bool dense) {
  (void)mw;
  ResLds w;
  uint32_t o = 0;
  w.dfa = o;
  o += pad16((uint32_t)(tb.S * tb.C * 2));
  w.bcls = o;
  o += 256;
  w.tinfo = o;
  o += 256 * 4;
  w.I = o;
  o += 32;
  w.acc_off = o;
  o += pad16((uint32_t)(tb.S + 1) * 4);
  w.acc_list = o;
  o += pad16((uint32_t)tb.n_acc);
  w.parse = o;
  w.pl = parse_lds(tb, o, dense);
  o += w.pl.total;
  w.live = o;  // the live sets as in global memory, 8 words per state
  o += pad16((uint32_t)(tb.S * 32));
  w.lanes = o;  // stack areas of the first kLaneSlots lanes of each wave
  o += (kWalkThreads / 64) * kLaneSlots * kFastLane * 2;
  w.umask = o;  // per work item: its residue bitmap word
  o += kMaxItems * 8;
  w.upre = o;   // prefix counts of residue spellings over the items
  o += (kMaxItems + 4) * 4;
  const uint32_t fixed = o + 64;
  w.block = (uint32_t)row_layout(tb).block;
  int g = kRowGroup < B ? kRowGroup : B;
  while (g > 1 && fixed + w.block * (uint32_t)g > kWalkLdsMax) --g;
  w.group = g;
  w.rows = o;
  o += w.block * (uint32_t)g;
  w.total = o;
  return w;
}

// The residue kernel's LDS: GOTO as the dense table when that still leaves
// room for the whole row group, else as the hash.
__host__ __device__ inline ResLds res_lds(const Tables& tb, int mw, int B) {
  const ResLds d = res_lds_with(tb, mw, B, true);
  if (d.group == (kRowGroup < B ? kRowGroup : B) && d.total + 64 <= kWalkLdsMax) return d;
  return res_lds_with(tb, mw, B, false);
}

// Everything the residue lanes share about the grammar (pointers into LDS).
template <int MW>
struct WalkShared {
  const Tables* tb;
  ParseTabs<true> pt;
  DfaView step;
  const uint32_t* tinfo;
  const uint32_t* I;
  const uint32_t* live;
  const uint32_t* acc_off;
  const uint8_t* acc_list;
  const uint16_t* pool;
};

// Verdict of one spelling left to the byte walk: byte 0 (continuing the
// pending lexeme, or ending it with the prologue's winner and starting a new
// one), then the byte-by-byte walk of the rest with emissions, overlay shifts
// and lexicon checks.  A lane whose stack area is too small hands its
// spelling to the slow path.  1 allowed, 0 rejected or handed over.
template <int MW>
__device__ __forceinline__ int residue_lane(const WalkShared<MW>& sh, const RowHeader& h, const uint8_t* rowblk,
                                            uint8_t* rw, const RowLayout& RL, uint32_t u, const uint4& rk,
                                            const uint4& tl, mptr<true, uint16_t> lane_area) {
  const Tables& tb = *sh.tb;
  const uint8_t* clsA = rowblk + sizeof(RowHeader);
  const uint8_t* clsW = clsA + pad16((uint32_t)tb.S);
  const uint32_t n = rk.w & 0xFFu;
  const uint64_t hb = (uint64_t)rk.x | (uint64_t)rk.y << 32;
  const uint32_t b0 = (uint32_t)(hb & 0xFF);
  const uint32_t c0 = sh.step.cls(b0);
  Slot sl;
  sl.fbase = h.slot[0];
  sl.hbase = h.slot[1];
  sl.hmask = h.slot[2];
  sl.restricted = h.slot[3];
  sl.nodes = h.slot[4];
  sl.pbase = h.slot[5];
  sl.pmask = h.slot[6];
  sl.sbase = h.slot[7];
  sl.smask = h.slot[8];
  RowCtx<true> rc;
  rc.tb = &tb;
  rc.pt = sh.pt;
  rc.bs = BaseStack<true>{sh.pool + h.stk_off, in_mem<true>((const uint16_t*)(rowblk + RL.win)), h.stk_depth,
                          h.stk_depth > (uint32_t)kWalkWin ? h.stk_depth - kWalkWin : 0u};
  rc.sl = sl;
  rc.tv = TermView{sh.tinfo, sh.I, h.R, sh.live, 8};
  rc.acc_off = sh.acc_off;
  rc.acc_list = sh.acc_list;
  rc.a2 = (const uint32_t*)(rw + RL.a2);
  rc.a2_stride = 8;
  rc.post = (const Post*)(rw + RL.post);
  rc.clsA = clsA;
  rc.clsW = clsW;
  rc.winner = h.wkind == 2 ? h.winner : -1;
  Lane<MW> ln;
  ln.k = 0;
  ln.m = 0;
  LexState lx;
  int q1 = sh.step.next((int)h.q, c0);
  const uint8_t* ct = clsA;
  bool dead = false;
  if (q1 != kDead) {  // byte 0 extends the pending lexeme
    ln.mode = 0;
    ln.t1 = -1;
    lx.len = h.rem_len + 1;
    lx.w = lx.len <= 8 ? (((uint64_t)h.rem_lo | (uint64_t)h.rem_hi << 32) | (uint64_t)b0 << (8 * h.rem_len)) : 0ull;
  } else {  // byte 0 ends it: its winner, then a new lexeme
    dead = h.wkind == 0;
    q1 = sh.step.next(kStart, c0);
    dead = dead || q1 == kDead;
    ln.mode = h.wkind == 2 ? 1 : 0;
    ln.t1 = h.wkind == 2 ? h.winner : -1;
    if (ln.mode == 1) ln.ph = reinterpret_cast<const uint4*>(rc.post)[2 * ln.t1];
    ct = h.wkind == 2 ? clsW : clsA;
    lx.len = 1;
    lx.w = b0;
  }
#pragma unroll
  for (int w = 0; w < MW; ++w) ln.acur[w] = ln.mode == 1 ? h.Aw[w] : h.A[w];
  const uint32_t f0 = dead ? 0u : (uint32_t)ct[q1];
  if (f0 == 0) return 0;  // byte 0 leaves no allowed or ignored terminal completable
  lx.need = sl.restricted != 0 && (f0 & 2u) ? 1u : 0u;
  lx.node = lx.need && lx.len > 8 ? lex_child(tb, sl, h.lexnode, b0) : kNoLex;
  SpellBytes byte_at;
  byte_at.win = hb >> 8;
  byte_at.lo0 = (uint64_t)tl.x | (uint64_t)tl.y << 32;
  byte_at.hi = (uint64_t)tl.z | (uint64_t)tl.w << 32;
  byte_at.ovf = tb.spell_tail + (rk.w >> 8);
  int ok = walk_bytes<true, MW>(rc, ln, q1, lx, 1u, n, byte_at, sh.step, lane_area, kFastLane, f0);
  if (ok < 0) {  // the lane's stack area is too small: hand over
    RowHeader* gh = (RowHeader*)rw;
    const uint32_t slot = atomicAdd(&gh->slow_count, 1u);
    if (slot < (uint32_t)kSlowCap) ((uint32_t*)(rw + RL.slow))[slot] = u;
    else atomicOr(&gh->wstat, GRID_ROW_OVERFLOW);
    ok = 0;
  }
  return ok;
}

// Bytes [s, s + 8) of the 24-byte window b0 b1 b2 (zero beyond it).
__device__ __forceinline__ uint64_t window8(uint64_t b0, uint64_t b1, uint64_t b2, uint32_t s) {
  const uint32_t w = s >> 3, sh = (s & 7u) * 8u;
  const uint64_t lo = w == 0 ? b0 : (w == 1 ? b1 : (w == 2 ? b2 : 0ull));
  const uint64_t hi = w == 0 ? b1 : (w == 1 ? b2 : 0ull);
  return sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
}

// Lexicon policy of a token judged with its own bytes: lexeme i of the
// class record (the pending bytes and the token's bytes before end 0, or the
// bytes between ends i-1 and i) and the trailing lexeme.  A lexeme starting
// in the start state at byte 0 or 1 is answered by the token-flag entry tf;
// others are looked up in the prefix and stride tables, and one that does not
// lie in the token's first 24 bytes is out of reach.  The pending bytes are
// known up to 8; beyond that the lexeme continues from the pending lexeme's
// trie node.  Plain scalar members only, so the policy lives in registers.
struct LexLane {
  const Tables* tb;
  Slot sl;
  uint64_t b0, b1, b2;  // token bytes 0..23, zero padded
  uint32_t n;           // token length
  uint32_t ends;        // lexeme ends (kClassMore: more than recorded)
  uint32_t pos;         // byte indices of ends 0, 1, 2 (8 bits each)
  uint64_t rem;         // pending bytes (first 8)
  uint32_t rem_len, lexnode;
  uint32_t tf;          // token-flag entry
  __device__ __forceinline__ uint32_t end_at(uint32_t i) const { return (pos >> (8 * i)) & 0xFFu; }
  __device__ __forceinline__ uint32_t span(uint32_t o, uint32_t e, bool pending) const {
    if (e > 24) return kLexOut;
    if (pending && rem_len > 0) {
      if (rem_len > 8) {  // continue from the pending lexeme's node
        uint32_t node = lexnode;
        for (uint32_t i = 0; i < e && node != kNoLex; ++i)
          node = lex_child(*tb, sl, node, (uint32_t)(window8(b0, b1, b2, i) & 0xFFu));
        return lex_flags_of(*tb, sl, node);
      }
      const uint32_t len = rem_len + e;
      if (len > 24) return kLexOut;
      const uint32_t s = 8u * rem_len;  // 8..64 bits: the token's bytes move up by rem_len
      const uint64_t c0 = rem | (s < 64 ? b0 << s : 0ull);
      const uint64_t c1 = (b0 >> (64 - s)) | (s < 64 ? b1 << s : 0ull);
      const uint64_t c2 = (b1 >> (64 - s)) | (s < 64 ? b2 << s : 0ull);
      return lex_flags_bytes(*tb, sl, c0, c1, c2, len);
    }
    return lex_flags_bytes(*tb, sl, window8(b0, b1, b2, o), window8(b0, b1, b2, o + 8), window8(b0, b1, b2, o + 16),
                           e - o);
  }
  __device__ __forceinline__ uint32_t word(uint32_t i) const {
    const int o = covered_start(pos, i, rem_len == 0);
    if (o >= 0) return ((tf >> (16 * o + 8)) & 0xFFu) << 8;
    return i == 0 ? span(0, end_at(0), true) : span(end_at(i - 1), end_at(i), false);
  }
  __device__ __forceinline__ uint32_t trail() const {
    if (ends > (uint32_t)kClassEnds) return kLexOut;
    const int o = covered_start(pos, ends, rem_len == 0);
    if (o >= 0) return (tf >> (16 * o)) & 0xFFu;
    return ends == 0 ? span(0, n, true) : span(end_at(ends - 1), n, false);
  }
};

// Verdict of one spelling of the residue bitmaps: for a spelling of the
// lexicon bitmap, its class cls (the class map's entry at its first id) is
// taken again with its own lexemes' lexicon flags (token-flag table, prefix and
// stride tables); the byte walk decides the rest.  1 allowed, 0 rejected or
// handed over.
template <int MW>
__device__ __forceinline__ int residue_token(const WalkShared<MW>& sh, const RowHeader& h, const uint8_t* rowblk,
                                             uint8_t* rw, const RowLayout& RL, uint32_t u, const uint4& rk,
                                             bool lexicon, uint32_t cls, mptr<true, uint16_t> lane_area) {
  const Tables& tb = *sh.tb;
  const uint32_t id0 = rk.z & 0x7FFFFFFFu;
  const uint32_t n = rk.w & 0xFFu;
  const uint4 tl = tb.spell_tail[u];
  if (lexicon) {
    const uint4 rec = tb.crec[h.cls_base + cls];
    LexLane lx;
    lx.tb = &tb;
    lx.sl = slot_of(h.slot);
    lx.n = n;
    lx.b0 = (uint64_t)rk.x | (uint64_t)rk.y << 32;
    lx.b1 = n > 8 ? (uint64_t)tl.x | (uint64_t)tl.y << 32 : 0ull;
    lx.b2 = n > 8 ? (uint64_t)tl.z | (uint64_t)tl.w << 32 : 0ull;
    lx.ends = rec.x & kClassEndsMask;
    lx.pos = rec.w;
    lx.rem = (uint64_t)h.rem_lo | (uint64_t)h.rem_hi << 32;
    lx.rem_len = h.rem_len;
    lx.lexnode = h.lexnode;
    lx.tf = tb.lex_token[(size_t)h.slot_id * tb.V + id0];
    const uint32_t v = class_verdict<MW, LexLane, false>(h, sh.I, sh.live, 8, sh.tinfo, sh.acc_off, sh.acc_list,
                                                         (const uint32_t*)(rw + RL.a2), 8, rec, lx);
    if (v == kVerdictAllow) return 1;
    if (v == kVerdictReject) return 0;
  }
  return residue_lane<MW>(sh, h, rowblk, rw, RL, u, rk, tl, lane_area);
}

// Sets the mask bit of every id that spells u (its alias ids).
__device__ inline void allow_spelling(const Tables& tb, uint32_t* mrow, uint32_t u, const uint4& rk) {
  if (!(rk.z >> 31)) {
    const uint32_t id = rk.z;
    atomicOr(mrow + (id >> 5), 1u << (id & 31u));
    return;
  }
  for (uint32_t a = tb.alias_off[u]; a < tb.alias_off[u + 1]; ++a) {
    const uint32_t id = (uint32_t)tb.alias_ids[a];
    atomicOr(mrow + (id >> 5), 1u << (id & 31u));
  }
}

// The rank-th set bit of m (rank < popcount(m)).
__device__ inline int nth_set_bit(uint64_t m, int rank) {
  int pos = 0;
#pragma unroll
  for (int w = 32; w >= 1; w >>= 1) {
    const uint64_t low = m & ((1ull << w) - 1ull);
    const int c = __popcll(low);
    if (rank >= c) {
      rank -= c;
      m >>= w;
      pos += w;
    } else {
      m = low;
    }
  }
  return pos;
}

// Persistent, one workgroup per compute unit.  For each group of rows that
// fits, a work item is one row against 64 consecutive spellings (one word of
// one of the row's residue bitmaps, byte-walk items first since they take
// longest); workgroup b takes items b, b + gridDim.x, ...
// and reads their words, then the set bits are packed into waves in
// spelling order, kWalkChunk byte-walk or kLexChunk lexicon spellings to a
// wave -- lexicographic neighbours walk alike, and a wave's time is the sum
// over its emission rounds of its slowest lane, so fewer lanes diverge less.  The grammar tables and the group's row blocks (header,
// trailing-flag tables, stack window) are staged in LDS only when the
// workgroup has residue spellings.  Each lane judges one spelling and sets
// the mask bits of its ids.
template <int MW>
__global__ __launch_bounds__(kWalkThreads) void residue_kernel(Tables tb, const uint16_t* __restrict__ pool,
                                                               uint32_t* __restrict__ mask, uint8_t* __restrict__ ws,
                                                               size_t rbytes, int B) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ int chunk_ctr;
  __shared__ uint32_t row_allowed[kRowGroup];  // the walk allowed a spelling of the group's row
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const ResLds WL = res_lds(tb, MW, B);
  const RowLayout RL = row_layout(tb);
  uint8_t* bcls = lds + WL.bcls;
  uint32_t* tinfo_s = (uint32_t*)(lds + WL.tinfo);
  uint32_t* I_s = (uint32_t*)(lds + WL.I);
  uint32_t* live_s = (uint32_t*)(lds + WL.live);
  uint64_t* umask_s = (uint64_t*)(lds + WL.umask);
  uint32_t* upre_s = (uint32_t*)(lds + WL.upre);
  const uint32_t* acc_off_s = (const uint32_t*)(lds + WL.acc_off);
  const uint8_t* acc_list_s = lds + WL.acc_list;
  uint8_t* rows_s = lds + WL.rows;
  // lanes kLaneSlots and above of a wave never judge a spelling (chunks are smaller)
  const mptr<true, uint16_t> lane_area =
      in_mem<true>((uint16_t*)(lds + WL.lanes) + ((tid >> 6) * kLaneSlots + (lane & (kLaneSlots - 1))) * kFastLane);
  uint8_t* rows = ws + kWsHead;
  const int nsub = (tb.U + 63) / 64;
  // the grammar tables go straight to LDS at once (direct global-to-LDS
  // loads, waited for at the first barrier that follows); the live sets are
  // staged as in global memory, 8 words per state
  {
    const StageRegion rg[10] = {{(const uint8_t*)tb.dfa, lds + WL.dfa, (uint32_t)(tb.S * tb.C * 2)},
                                {tb.bclass, bcls, 256u},
                                {(const uint8_t*)tb.acc_off, lds + WL.acc_off, (uint32_t)(tb.S + 1) * 4},
                                {tb.acc_list, lds + WL.acc_list, (uint32_t)tb.n_acc},
                                {(const uint8_t*)tb.live, (uint8_t*)live_s, (uint32_t)tb.S * 32u},
                                {(const uint8_t*)tb.term_info, (uint8_t*)tinfo_s, (uint32_t)tb.T * 4u},
                                parse_region(tb, lds, WL.pl, 0),
                                parse_region(tb, lds, WL.pl, 1),
                                parse_region(tb, lds, WL.pl, 2),
                                parse_region(tb, lds, WL.pl, 3)};
    dma_regions<10>(rg, tid, kWalkThreads);
  }
  if (tid < 8) I_s[tid] = tb.ign[tid];
  for (int g0 = 0; g0 < B; g0 += WL.group) {
    const int gr = min(WL.group, B - g0);
    const int items = 2 * gr * nsub;  // walk items of the group's rows first, then lexicon items
    const int mine = items > (int)blockIdx.x ? (items - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x : 0;
    bool blocks = false;  // the group's row blocks are in LDS
    if (tid < kRowGroup) row_allowed[tid] = 0u;
    for (int k0 = 0; k0 < mine; k0 += kMaxItems) {
      const int n_it = min(kMaxItems, mine - k0);
      // this thread's item word, loaded before the wait for the table copies
      static_assert(kMaxItems == kWalkThreads, "one item word per thread");
      uint64_t uw = 0ull;
      if (tid < n_it) {
        const int j = (int)blockIdx.x + (k0 + tid) * (int)gridDim.x;
        const int lex = j >= gr * nsub ? 1 : 0, jr = j - lex * gr * nsub;
        const int r = jr / nsub;
        const uint8_t* rw = rows + (size_t)(g0 + r) * rbytes;
        const uint32_t v = ((const RowHeader*)rw)->valid;
        const uint64_t word = ((const uint64_t*)(rw + RL.rbits))[(lex ? 0 : nsub) + jr - r * nsub];
        uw = v == kRowValid ? word : 0ull;
      }
      dma_wait();
      __syncthreads();  // the previous round is done with umask_s / upre_s; the tables are in LDS
      if (tid < n_it) umask_s[tid] = uw;
      if (tid == 0) chunk_ctr = 0;
      __syncthreads();
      if (tid < 64) {  // prefix counts of set bits over the items (one wave)
        const int per = (n_it + 63) / 64;
        uint32_t sum = 0;
        for (int i = 0; i < per; ++i) {
          const int t = lane * per + i;
          if (t < n_it) sum += (uint32_t)__popcll(umask_s[t]);
        }
        uint32_t incl = sum;
#pragma unroll
        for (int d = 1; d < 64; d <<= 1) {
          const uint32_t x = __shfl_up(incl, d);
          if (lane >= d) incl += x;
        }
        uint32_t run = incl - sum;
        for (int i = 0; i < per; ++i) {
          const int t = lane * per + i;
          if (t < n_it) {
            upre_s[t] = run;
            run += (uint32_t)__popcll(umask_s[t]);
          }
        }
        if (lane == 63) upre_s[n_it] = incl;
      }
      __syncthreads();
      const int n_und = (int)upre_s[n_it];
      if (n_und == 0) continue;  // uniform
      if (!blocks) {  // the rows' blocks, two 16-byte chunks per thread in flight at a time
        const uint32_t n16 = WL.block / 16u, tot16 = (uint32_t)gr * n16;
        for (uint32_t i = tid; i < tot16; i += 2u * kWalkThreads) {
          const uint32_t i2 = i + kWalkThreads;
          const uint32_t r = i / n16, r2 = i2 / n16;
          const uint4 v = reinterpret_cast<const uint4*>(rows + (size_t)(g0 + r) * rbytes)[i - r * n16];
          uint4 v2 = make_uint4(0, 0, 0, 0);
          if (i2 < tot16) v2 = reinterpret_cast<const uint4*>(rows + (size_t)(g0 + r2) * rbytes)[i2 - r2 * n16];
          reinterpret_cast<uint4*>(rows_s)[i] = v;
          if (i2 < tot16) reinterpret_cast<uint4*>(rows_s)[i2] = v2;
        }
        blocks = true;
      }
      __syncthreads();
      const ParseTabs<true> pt = lds_parse(tb, lds, WL.pl);
      const DfaView step{(const uint16_t*)(lds + WL.dfa), bcls, tb.C};
      const WalkShared<MW> sh{&tb, pt, step, tinfo_s, I_s, live_s, acc_off_s, acc_list_s, pool};
      // positions [0, n_wpos) belong to byte-walk items (they come first), the
      // rest to lexicon items; a wave takes kWalkChunk walk positions or
      // kLexChunk lexicon positions at a time (fewer lanes, less divergence)
      const int t_lex0 = min(max((gr * nsub - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x - k0, 0), n_it);
      const int n_wpos = (int)upre_s[t_lex0];
      const int nwc = (n_wpos + kWalkChunk - 1) / kWalkChunk;
      for (;;) {
        const int c = wave_grab(&chunk_ctr);
        int pos;
        bool in;
        if (c < nwc) {
          pos = c * kWalkChunk + lane;
          in = lane < kWalkChunk && pos < n_wpos;
        } else {
          if (n_wpos + (c - nwc) * kLexChunk >= n_und) break;
          pos = n_wpos + (c - nwc) * kLexChunk + lane;
          in = lane < kLexChunk && pos < n_und;
        }
        if (in) {
          // the item holding position pos: last t with upre_s[t] <= pos
          int lo = 0, hi = n_it - 1;
          while (lo < hi) {
            const int mid = (lo + hi + 1) >> 1;
            if ((int)upre_s[mid] <= pos) lo = mid;
            else hi = mid - 1;
          }
          const int bit = nth_set_bit(umask_s[lo], pos - (int)upre_s[lo]);
          const int j = (int)blockIdx.x + (k0 + lo) * (int)gridDim.x;
          const int lex = j >= gr * nsub ? 1 : 0, jr = j - lex * gr * nsub;
          const int r = jr / nsub;
          const uint32_t u = (uint32_t)((jr - r * nsub) * 64 + bit);
          const uint8_t* rowblk = rows_s + (size_t)r * WL.block;
          uint8_t* rw = rows + (size_t)(g0 + r) * rbytes;
          const uint4 rk = tb.spell_rec[u];
          // a lexicon spelling's class: the class map at its first id (its
          // aliases share it)
          const uint32_t cls =
              lex ? (uint32_t)tb.cmap[(size_t)((const RowHeader*)rowblk)->q * tb.V + (rk.z & 0x7FFFFFFFu)] : 0u;
          const RowHeader& hh = *(const RowHeader*)rowblk;
          // a lexicon spelling of a CI class also goes to the row's claimed CI-words entry
          const bool ci_tok = lex && hh.ci_claim >= 0 && ci_class(tb.crec[hh.cls_base + cls].x);
          if (residue_token<MW>(sh, hh, rowblk, rw, RL, u, rk, lex != 0, cls, lane_area) > 0) {
            allow_spelling(tb, mask + (size_t)(g0 + r) * tb.W, u, rk);
            if (ci_tok)
              allow_spelling(tb, (uint32_t*)(tb.ci_cache + (size_t)hh.ci_claim * tb.ci_stride + kCiHeader), u, rk);
            row_allowed[r] = 1u;
          }
        }
      }
    }
    __syncthreads();  // every wave is done with the group: one header store per row that got a token
    if (tid < gr && row_allowed[tid]) ((RowHeader*)(rows + (size_t)(g0 + tid) * rbytes))->nonempty = 1u;
  }
  dma_wait();  // a workgroup without items still has its table copies in flight
}

// ---------------------------------------------------------------- finalize
// One workgroup per row.  Spellings the residue walk handed over (their lane
// stack area was too small) are walked again from the row's configuration
// with a large stack area per thread in the workspace, reading the tables
// from global memory; then the row status is written.
template <int MW>
__global__ __launch_bounds__(kBlock) void finalize_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                          const uint16_t* __restrict__ pool,
                                                          uint32_t* __restrict__ mask, uint8_t* __restrict__ ws,
                                                          size_t rbytes, int32_t* __restrict__ status) {
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  uint8_t* rw = ws + kWsHead + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  const RowLayout RL = row_layout(tb);
  if (hdr->valid == kRowCached) {  // served from the mask cache by the prologue
    if (threadIdx.x == 0 && status) status[row] = hdr->pstat;
    return;
  }
  const bool valid = hdr->valid == kRowValid;
  const uint32_t count = valid ? min(hdr->slow_count, (uint32_t)kSlowCap) : 0u;
  __shared__ uint32_t I_s[8];
  __shared__ int slow_ok;
  if (tid == 0) slow_ok = 0;
  if (count > 0) {  // uniform
    if (tid < 8) I_s[tid] = tb.ign[tid];
    const ParseTabs<false> pt = global_parse(tb);  // rare: tables stay in global memory
    __syncthreads();
    if (tid < kSlowThreads) {
      const grid_config cfg = cfgs[row];
      RowCtx<false> rc;
      rc.tb = &tb;
      rc.pt = pt;
      rc.bs = BaseStack<false>{pool + cfg.stk_off, nullptr, cfg.stk_depth, cfg.stk_depth};
      rc.sl = load_slot(tb, cfg.slot);
      rc.tv = TermView{tb.term_info, I_s, hdr->R, tb.live, 8};
      rc.acc_off = tb.acc_off;
      rc.acc_list = tb.acc_list;
      rc.a2 = (const uint32_t*)(rw + RL.a2);
      rc.a2_stride = 8;
      rc.post = (const Post*)(rw + RL.post);
      rc.clsA = nullptr;
      rc.clsW = nullptr;
      rc.winner = -1;
      uint16_t* ov = (uint16_t*)(rw + RL.slow_ov) + tid * kSlowLane;
      const DfaView step{tb.dfa, tb.bclass, tb.C};
      LexState lex0;
      lex0.len = cfg.flags & 1u ? 0u : cfg.rem_len;
      lex0.node = cfg.lexnode;
      lex0.need = rc.sl.restricted != 0 ? 1u : 0u;
      lex0.w = 0;
      for (int k = 0; k < 8; ++k) lex0.w |= (uint64_t)cfg.rem_head[k] << (8 * k);
      for (uint32_t k = tid; k < count; k += kSlowThreads) {
        const uint32_t su = ((const uint32_t*)(rw + RL.slow))[k];
        Lane<MW> ln;
        ln.mode = 0;
        ln.t1 = -1;
        ln.k = 0;
        ln.m = 0;
#pragma unroll
        for (int w = 0; w < MW; ++w) ln.acur[w] = hdr->A[w];
        const uint32_t base = tb.spell_off[su];
        auto byte_at = [&](uint32_t i) -> uint32_t { return tb.spell_bytes[base + i]; };
        const int ok = walk_bytes<false, MW>(rc, ln, cfg.q, lex0, 0u, tb.spell_off[su + 1] - base, byte_at, step,
                                             ov, kSlowLane, 1u);
        if (ok > 0) {
          const uint4 rk = tb.spell_rec[su];
          allow_spelling(tb, mask + (size_t)row * tb.W, su, rk);
          if (hdr->ci_claim >= 0) {  // a CI-class spelling also goes to the row's claimed entry
            const uint32_t cls = tb.cmap[(size_t)cfg.q * tb.V + (rk.z & 0x7FFFFFFFu)];
            if (ci_class(tb.crec[hdr->cls_base + cls].x))
              allow_spelling(tb, (uint32_t*)(tb.ci_cache + (size_t)hdr->ci_claim * tb.ci_stride + kCiHeader), su, rk);
          }
          slow_ok = 1;
        } else if (ok < 0) {
          atomicOr(&hdr->wstat, GRID_ROW_OVERFLOW);
        }
      }
    }
  }
  __syncthreads();
  if (tid == 0) {
    int32_t st;
    if (valid) {
      st = hdr->pstat | hdr->wstat;
      if (hdr->slow_count > (uint32_t)kSlowCap) st |= GRID_ROW_OVERFLOW;
      if (!hdr->nonempty && !slow_ok && !hdr->eos_ok) st |= GRID_ROW_EMPTY;
    } else {
      st = hdr->pstat | GRID_ROW_BAD_CONFIG;
    }
    if (status) status[row] = st;
    hdr->fstat = st;
    if (valid && hdr->ci_claim >= 0) {  // publish the row's CI-words entry, or give the slot back
      uint32_t* e = (uint32_t*)(tb.ci_cache + (size_t)hdr->ci_claim * tb.ci_stride);
      __threadfence();
      __hip_atomic_store(e, st == GRID_ROW_OK ? 2u : 0u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// Mask cache write-back: each row that claimed an entry in the prologue
// copies its finished mask row, EOS flag and status into it, then publishes
// it (a device-scope fence orders the copy before the state word).
__global__ __launch_bounds__(kBlock) void cache_publish_kernel(Tables tb, const uint32_t* __restrict__ mask,
                                                               const uint8_t* __restrict__ ws, size_t rbytes) {
  const int row = blockIdx.x;
  const RowHeader* hdr = (const RowHeader*)(ws + kWsHead + (size_t)row * rbytes);
  if (hdr->valid != kRowValid || hdr->cache_slot < 0) return;  // uniform
  CacheEntry* e = (CacheEntry*)(tb.cache + (size_t)hdr->cache_slot * tb.cache_stride);
  uint32_t* dst = (uint32_t*)(e + 1);
  const uint32_t* src = mask + (size_t)row * tb.W;
  for (int i = threadIdx.x; i < tb.W; i += kBlock) dst[i] = src[i];
  if (threadIdx.x == 0) {
    e->eos = hdr->eos_ok;
    e->status = (uint32_t)hdr->fstat;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    __threadfence();
    __hip_atomic_store(&e->state, 2u, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Empties a mask cache: every entry's state word to 0.
__global__ __launch_bounds__(kBlock) void cache_clear_kernel(uint8_t* cache, uint32_t n, uint32_t stride) {
  for (uint32_t i = blockIdx.x * kBlock + threadIdx.x; i < n; i += gridDim.x * kBlock)
    ((CacheEntry*)(cache + (size_t)i * stride))->state = 0u;
}

// ------------------------------------------------------------------- apply
// Each thread covers 8 consecutive logits of one row; the mask byte for them
// comes from one word.  An aligned group takes 16-byte stores (read first
// when it keeps entries, whose bits are written back unchanged); a group at
// a ragged row end or in an unaligned row is written logit by logit.
template <typename T>
__global__ __launch_bounds__(kBlock) void apply_kernel(const uint32_t* __restrict__ mask, T* logits, int B,
                                                       int V, int W, int64_t stride, uint32_t neg_inf_bits,
                                                       bool vec_ok) {
  // row blockIdx.y; groups of 8 logits along it, grid-stride in x
  const int groups = (V + 7) >> 3;
  const int row = (int)blockIdx.y;
  (void)B;
  for (int grp = (int)(blockIdx.x * kBlock + threadIdx.x); grp < groups; grp += (int)(gridDim.x * kBlock)) {
    const int col = grp * 8;
    const uint32_t bits = (mask[(size_t)row * W + (col >> 5)] >> (col & 31)) & 0xFFu;
    if (bits == 0xFFu) continue;
    T* p = logits + (int64_t)row * stride + col;
    if (col + 8 <= V && vec_ok) {  // whole group: 16-byte stores, the kept logits read back unchanged
      if (sizeof(T) == 2) {
        uint4 v = bits ? *reinterpret_cast<const uint4*>(p) : make_uint4(0, 0, 0, 0);
        uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          const uint32_t lo = (bits >> (2 * k)) & 1u ? w[k] & 0xFFFFu : neg_inf_bits;
          const uint32_t hi = (bits >> (2 * k + 1)) & 1u ? w[k] & 0xFFFF0000u : neg_inf_bits << 16;
          w[k] = lo | hi;
        }
        *reinterpret_cast<uint4*>(p) = make_uint4(w[0], w[1], w[2], w[3]);
      } else {
        uint4 v0 = make_uint4(0, 0, 0, 0), v1 = v0;
        if (bits & 0x0Fu) v0 = reinterpret_cast<const uint4*>(p)[0];
        if (bits & 0xF0u) v1 = reinterpret_cast<const uint4*>(p)[1];
        const uint32_t w[8] = {v0.x, v0.y, v0.z, v0.w, v1.x, v1.y, v1.z, v1.w};
        uint32_t o[8];
#pragma unroll
        for (int k = 0; k < 8; ++k) o[k] = (bits >> k) & 1u ? w[k] : neg_inf_bits;
        reinterpret_cast<uint4*>(p)[0] = make_uint4(o[0], o[1], o[2], o[3]);
        reinterpret_cast<uint4*>(p)[1] = make_uint4(o[4], o[5], o[6], o[7]);
      }
      continue;
    }
    for (int j = 0; j < 8 && col + j < V; ++j) {
      if (!((bits >> j) & 1u)) {
        if (sizeof(T) == 2) reinterpret_cast<uint16_t*>(p)[j] = (uint16_t)neg_inf_bits;
        else reinterpret_cast<uint32_t*>(p)[j] = neg_inf_bits;
      }
    }
  }
}

// ------------------------------------------------------------------ accept
// The whole stack stk[0, d) as a read-only base for simulations: in LDS it
// is the window, in global memory the pool.
template <bool L>
__device__ inline BaseStack<L> whole_stack(mptr<L, uint16_t> stk, uint32_t d) {
  if constexpr (L) return BaseStack<L>{nullptr, stk, d, 0u};
  else return BaseStack<L>{stk, nullptr, d, d};
}

// Reduce chain of terminal x on the stack stk[0, d), pushes above d (the
// stack below stays as it is).  1 shift, 2 accept (x is the end of input), 0
// error, -1 capacity.  With commit, a shift makes the chain's result the
// stack: the pushed states move down onto the popped entries, then x's
// shift target goes on top (so a winner costs one chain, not two).
template <bool L, int MW>
__device__ int chain_shift(const ParseTabs<L>& pt, mptr<L, uint16_t> stk, uint32_t& d, uint32_t cap, int x,
                           bool commit, uint32_t& lo_mod) {
  if (d >= cap) return -1;
  const BaseStack<L> bs = whole_stack<L>(stk, d);
  const mptr<L, uint16_t> tmp = stk + d;
  const int tmpcap = (int)(cap - d);
  const uint32_t w = (uint32_t)x >> 5, bit = 1u << (x & 31);
  uint32_t k = d;
  int m = 0, t = 0;
  uint32_t s = stack_at_top<L>(bs, k, m, tmp, 0, tmp), below = kNoState;
  for (int guard = 0; guard < kGuard; ++guard) {
    const uint32_t a = action_of<L, MW>(pt, s, w, bit);
    if (a >= kActShiftP) {
      if (a != kActShiftP) return 0;
      if (x == pt.T) return 2;
      if (commit) {
        for (int i = 0; i < t; ++i) stk[k + (uint32_t)i] = tmp[i];  // k <= d: a forward move is safe
        lo_mod = min(lo_mod, k);
        d = k + (uint32_t)t;
        if (d >= cap) return -1;
        stk[d++] = shift_target<L, MW>(pt, s, x, true);  // the LALR stack
      }
      return 1;
    }
    const uint32_t len = a >> 16;
    if (!pop_len(len, k, m, t)) return 0;
    const uint32_t sb = goto_source<L>(bs, len, s, below, k, m, tmp, t, tmp);
    const uint16_t g = goto_of<L>(pt, sb, a & 0xFFFFu);
    if (g == kNoGoto) return 0;
    if (t >= tmpcap) return -1;
    tmp[t++] = g;
    below = sb;
    s = g;
  }
  return -1;
}

// The lexer tables an advance reads (global memory, or their LDS copies).
struct LexPtrs {
  const uint16_t* dfa;
  const uint8_t* bclass;
  const uint32_t* term_info;
  const uint32_t* acc_off;
  const uint8_t* acc_list;
  const uint32_t* live;
};

struct AccLex {  // a row's lexer side: DFA state, lexicon node, pending lexeme
  uint32_t q, lex, rem;
  uint8_t head[8];
};

// One row's advance by token tok (section 6.1, per-token step 7) on the stack
// stk[0, d) of capacity cap, with the LR tables pt; lo_mod falls to the
// lowest stack index the advance rewrites (entries below it are unchanged).  The token's bytes go
// through the lexer with maximal munch; a byte that kills the DFA emits the
// pending lexeme as the highest-priority candidate that is ignored or shifts
// and passes its category's lexicon, and a shifted terminal runs its reduce
// chain on the stack.  The new pending lexeme must still complete to an
// allowed or ignored terminal (Definition 2).  The end-of-sequence token is
// accepted when the end-of-sequence gate holds (section 3.2).  Returns the
// row status; with GRID_ROW_OK, d and lx are the new configuration's.
template <bool L, int MW>
__device__ __forceinline__ int advance_row(const Tables& tb, const LexPtrs lp, const ParseTabs<L>& pt, const Slot& sl,
                           mptr<L, uint16_t> stk, uint32_t& d, uint32_t cap, int tok, AccLex& lx,
                           uint32_t& lo_mod) {
  auto ignored = [&](int t) { return (lp.term_info[t] & 1u) != 0; };
  auto restricted_cat = [&](int t) -> int {  // category the row's lexicon restricts, or -1
    const uint32_t c = (lp.term_info[t] >> 8) & 0xFFu;
    return c != 0xFFu && ((sl.restricted >> c) & 1u) ? (int)c : -1;
  };
  // can terminal t be shifted from the stack now (reduce chain only, pushes
  // above the stack, which stays as it is)?
  // 1 shift, 2 accept (the end of input), 0 error, -1 capacity
  auto shifts = [&](int t) -> int { return chain_shift<L, MW>(pt, stk, d, cap, t, false, lo_mod); };
  // the pending lexeme's winner in state q (lexicon node lex), its reduce
  // chain and shift applied to the stack when it is not ignored: -1 none,
  // else the terminal; capacity problems surface as -2
  auto winner = [&]() -> int {
    for (uint32_t j = lp.acc_off[lx.q]; j < lp.acc_off[lx.q + 1]; ++j) {
      const int t = lp.acc_list[j];
      const int c = restricted_cat(t);
      if (c >= 0 && !((lex_flags_of(tb, sl, lx.lex) >> (8 + c)) & 1u)) continue;
      if (ignored(t)) return t;
      const int r = chain_shift<L, MW>(pt, stk, d, cap, t, true, lo_mod);
      if (r < 0) return -2;
      if (r == 1) return t;
    }
    return -1;
  };
  if (tok == tb.eos_id) {  // the configuration itself stays as it is
    int ok = 0;
    if (lx.rem == 0) {
      ok = shifts(tb.T) == 2;
    } else {
      const int w = winner();
      if (w == -2) return GRID_ROW_OVERFLOW;
      if (w >= 0) ok = shifts(tb.T) == 2;
    }
    return ok ? GRID_ROW_FINISHED : GRID_ROW_NOT_VIABLE;
  }
  const uint32_t su = tb.spell_of_id[tok];
  if (su == 0xFFFFFFFFu) return GRID_ROW_NOT_VIABLE;  // special or empty token
  const uint32_t b0 = tb.spell_off[su], n = tb.spell_off[su + 1] - b0;
  for (uint32_t i = 0; i < n; ++i) {
    const uint32_t b = tb.spell_bytes[b0 + i];
    const int nq = lp.dfa[lx.q * tb.C + lp.bclass[b]];
    if (nq != kDead) {
      lx.q = (uint32_t)nq;
      lx.lex = lex_child(tb, sl, lx.lex, b);
      if (lx.rem < 8) lx.head[lx.rem] = (uint8_t)b;
      ++lx.rem;
      continue;
    }
    // b kills the pending lexeme: emit it
    if (lx.rem == 0 || lp.acc_off[lx.q + 1] == lp.acc_off[lx.q]) return GRID_ROW_NOT_VIABLE;
    const int w = winner();
    if (w == -2) return GRID_ROW_OVERFLOW;
    if (w < 0) return GRID_ROW_NOT_VIABLE;
    const int q1 = lp.dfa[kStart * tb.C + lp.bclass[b]];
    if (q1 == kDead) return GRID_ROW_NOT_VIABLE;
    lx.q = (uint32_t)q1;
    lx.lex = lex_child(tb, sl, 0u, b);
    lx.rem = 1;
    lx.head[0] = (uint8_t)b;
    for (int k = 1; k < 8; ++k) lx.head[k] = 0;
  }
  if (lx.rem == 0) return GRID_ROW_OK;
  // Definition 2 for the pending lexeme
  const uint32_t* lv = lp.live + (size_t)lx.q * 8;
  for (int wd = 0; wd < 8; ++wd) {
    for (uint32_t bits = lv[wd]; bits != 0u; bits &= bits - 1u) {  // live terminals in id order
      const int t = wd * 32 + __builtin_ctz(bits);
      if (t >= tb.T) break;
      const int c = restricted_cat(t);
      if (c >= 0 && !((lex_flags_of(tb, sl, lx.lex) >> c) & 1u)) continue;
      if (ignored(t)) return GRID_ROW_OK;
      const int r = shifts(t);
      if (r < 0) return GRID_ROW_OVERFLOW;
      if (r == 1) return GRID_ROW_OK;
    }
  }
  return GRID_ROW_NOT_VIABLE;
}

// LDS bytes of the lexer tables an accept workgroup stages beside the LR
// tables and the stack: DFA, byte classes, terminal info, accept lists, live
// sets (offsets from the start of the area).
struct AccLexLds {
  uint32_t dfa, bclass, tinfo, acc_off, acc_list, live, total;
};
__host__ __device__ inline AccLexLds accept_lex_lds(const Tables& tb) {
  AccLexLds L;
  uint32_t o = 0;
  L.dfa = o;
  o += pad16((uint32_t)(tb.S * tb.C * 2));
  L.bclass = o;
  o += 256;
  L.tinfo = o;
  o += pad16((uint32_t)tb.T * 4u);
  L.acc_off = o;
  o += pad16((uint32_t)(tb.S + 1) * 4u);
  L.acc_list = o;
  o += pad16((uint32_t)tb.n_acc);
  L.live = o;
  o += pad16((uint32_t)tb.S * 32u);
  L.total = o;
  return L;
}
constexpr uint32_t kAcceptLdsMax = 152 * 1024;

constexpr uint32_t kAccStack = 8192;  // stack entries an accept workgroup keeps in LDS

__host__ __device__ inline uint32_t accept_stack_cap(uint32_t cap) { return cap < kAccStack ? cap : kAccStack; }

// Device incremental advance: one workgroup per row.  The LR tables and the
// row's stack are staged in LDS and one thread advances the row there (the
// chain of dependent table reads is the cost, so every read is an LDS read).
// Every row's output is self-contained, whatever its status: the input stack
// is copied to the row's own area pool_out + b * cap (checking every entry is
// an LR state) and the configuration written to cfg_out points there; an
// advance then rewrites only the entries from the lowest one it changed.  A
// stack that outgrows the LDS area while cap allows more is advanced again
// from the start, by the same routine, on that global copy with the tables in
// global memory; so is every row when the LR tables are too large to stage
// (use_lds = 0).  A row whose stack does not fit cap gets depth 0 (a
// configuration every call rejects).
//
// In place (inplace = 1; cfg_out == cfgs, pool_out == pool): row b's stack
// lives in pool[b * cap, (b + 1) * cap) and is its persistent arena -- the
// entries below the lowest one a step rewrites are neither copied nor
// written, the rewritten ones are written back from LDS, and, with hash, the
// rolling hash of every rewritten entry is recomputed from its parent's (one
// hash per pushed node).  A row that is not advanced keeps its stack and
// configuration untouched; a stack too deep for the LDS area is reported as
// an overflow (the out-of-place call handles it).
template <int MW>
__global__ __launch_bounds__(kBlock) void accept_kernel(Tables tb, const grid_config* cfgs, const uint16_t* pool,
                                                        const int32_t* __restrict__ tokens, grid_config* cfg_out,
                                                        uint16_t* pool_out, uint64_t* hash, uint32_t cap,
                                                        int32_t* status, int use_lds, int use_lex, int inplace,
                                                        int tok_stride) {
  extern __shared__ __align__(16) uint8_t alds[];
  __shared__ int s_st, s_bad;
  __shared__ uint32_t s_d, s_lo;
  const int row = (int)blockIdx.x, tid = (int)threadIdx.x;
  const grid_config cfg = cfgs[row];
  const int tok = tokens[(size_t)row * tok_stride];
  const uint32_t d0 = cfg.stk_depth;
  uint16_t* out_stk = pool_out + (size_t)row * cap;
  const bool copyable = d0 >= 1 && d0 <= cap && (!inplace || cfg.stk_off == (uint32_t)row * cap);  // uniform
  bool bad = !copyable || cfg.q >= (uint32_t)tb.S || cfg.q == (uint32_t)kDead || cfg.slot >= (uint32_t)tb.n_slots ||
             tok < 0 || tok >= tb.V;
  Slot sl{};
  if (!bad) {
    sl = load_slot(tb, (int)cfg.slot);
    bad = cfg.lexnode != kNoLex && cfg.lexnode >= sl.nodes;
  }
  if (tid == 0) s_bad = 0;
  const ParseLds PL = prologue_parse_lds(tb);
  const uint32_t lcap = accept_stack_cap(cap);
  const mptr<true, uint16_t> stk_l = in_mem<true>((uint16_t*)(alds + PL.total));
  if (use_lds && !bad) {
    const StageRegion rg[4] = {parse_region(tb, alds, PL, 0), parse_region(tb, alds, PL, 1),
                               parse_region(tb, alds, PL, 2), parse_region(tb, alds, PL, 3)};
    dma_regions<4>(rg, tid, kBlock);
  }
  // the lexer tables too when they fit: every byte step is then an LDS read
  const AccLexLds XL = accept_lex_lds(tb);
  uint8_t* xl = alds + PL.total + pad16(lcap * 2u);
  LexPtrs lp{tb.dfa, tb.bclass, tb.term_info, tb.acc_off, tb.acc_list, tb.live};
  if (use_lds && use_lex && !bad) {
    const StageRegion rg[6] = {{(const uint8_t*)tb.dfa, xl + XL.dfa, (uint32_t)(tb.S * tb.C * 2)},
                               {tb.bclass, xl + XL.bclass, 256u},
                               {(const uint8_t*)tb.term_info, xl + XL.tinfo, (uint32_t)tb.T * 4u},
                               {(const uint8_t*)tb.acc_off, xl + XL.acc_off, (uint32_t)(tb.S + 1) * 4u},
                               {tb.acc_list, xl + XL.acc_list, (uint32_t)tb.n_acc},
                               {(const uint8_t*)tb.live, xl + XL.live, (uint32_t)tb.S * 32u}};
    dma_regions<6>(rg, tid, kBlock, 1000u);
    lp = LexPtrs{(const uint16_t*)(xl + XL.dfa), xl + XL.bclass, (const uint32_t*)(xl + XL.tinfo),
                 (const uint32_t*)(xl + XL.acc_off), xl + XL.acc_list, (const uint32_t*)(xl + XL.live)};
  }
  const bool fits = use_lds && !bad && d0 < lcap;  // uniform
  dma_wait();
  __syncthreads();  // s_bad is cleared, the tables are in LDS
  if (copyable) {  // the input stack to the row's output area (and to LDS), entries checked
    for (uint32_t i = (uint32_t)tid; i < d0; i += kBlock) {
      const uint16_t v = pool[cfg.stk_off + i];
      if (v >= (uint32_t)tb.NS) s_bad = 1;
      if (!inplace) out_stk[i] = v;
      if (fits) stk_l[i] = v;
    }
  }
  __syncthreads();
  bad = bad || s_bad != 0;  // uniform
  grid_config out = cfg;
  if (!inplace) {
    if (copyable) out.stk_off = (uint32_t)row * cap;
    else out.stk_depth = 0;
  }
  if (bad) {
    if (tid == 0) {
      if (!inplace) cfg_out[row] = out;
      if (status) status[row] = GRID_ROW_BAD_CONFIG;
    }
    return;
  }
  AccLex lx;
  lx.q = cfg.q;
  lx.lex = cfg.lexnode;
  lx.rem = (cfg.flags & 1u) ? 0u : cfg.rem_len;
  for (int k = 0; k < 8; ++k) lx.head[k] = lx.rem > 0 ? cfg.rem_head[k] : 0;
  int st = -1;  // -1: not advanced in LDS
  uint32_t d = d0, lo = d0;
  if (tid == 0) {
    if (fits) {
      st = advance_row<true, MW>(tb, lp, lds_parse(tb, alds, PL), sl, stk_l, d, lcap, tok, lx, lo);
      if (st == GRID_ROW_OVERFLOW && lcap < cap) st = -1;
    }
    if (inplace && st == -1) st = GRID_ROW_OVERFLOW;  // in place, only the LDS route
    s_st = st;
    s_d = d;
    s_lo = lo;
  }
  __syncthreads();
  if (s_st == GRID_ROW_OK) {  // the entries the advance rewrote
    for (uint32_t i = s_lo + (uint32_t)tid; i < s_d; i += kBlock) out_stk[i] = stk_l[i];
  } else if (s_st == -1 && tid == 0) {  // the global route, from the start, on the output copy
    lx.q = cfg.q;
    lx.lex = cfg.lexnode;
    lx.rem = (cfg.flags & 1u) ? 0u : cfg.rem_len;
    for (int k = 0; k < 8; ++k) lx.head[k] = lx.rem > 0 ? cfg.rem_head[k] : 0;
    d = d0;
    lo = d0;
    const LexPtrs lg{tb.dfa, tb.bclass, tb.term_info, tb.acc_off, tb.acc_list, tb.live};
    st = advance_row<false, MW>(tb, lg, global_parse(tb), sl, out_stk, d, cap, tok, lx, lo);
    if (st != GRID_ROW_OK)  // a refused token leaves the row's input stack in its area
      for (uint32_t i = lo; i < d0; ++i) out_stk[i] = pool[cfg.stk_off + i];
  }
  if (tid != 0) return;
  if (st == GRID_ROW_OK && hash) {  // rolling hashes of the rewritten entries, each from its parent's
    const uint32_t off = out.stk_off;
    uint64_t h = hash[off + lo - 1];  // lo >= 1: the bottom entry is never popped
    for (uint32_t i = lo; i < d; ++i) {
      const uint32_t sv = fits ? (uint32_t)stk_l[i] : (uint32_t)out_stk[i];
      h = node_hash(h, sv, tb.state_sym[sv]);
      hash[off + i] = h;
    }
  }
  if (inplace && st != GRID_ROW_OK) {
    if (status) status[row] = st;
    return;
  }
  if (st == GRID_ROW_OK) {
    out.stk_depth = d;
    out.lexnode = lx.lex;
    out.q = (uint16_t)lx.q;
    out.flags = lx.rem == 0 ? 1u : 0u;
    out.rem_len = lx.rem;
    for (int k = 0; k < 8; ++k) out.rem_head[k] = lx.head[k];
  }
  cfg_out[row] = out;
  if (status) status[row] = st;
}

// Rolling hash of every stack entry of every row (one thread per row: each
// entry's hash needs its parent's): entry 0 is the root (hash 0), entry i > 0
// hashes the one below it, its LR state and that state's accessing symbol.
__global__ __launch_bounds__(64) void stack_hash_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                       const uint16_t* __restrict__ pool, uint64_t* __restrict__ hash,
                                                       int B) {
  const int row = (int)(blockIdx.x * 64u + threadIdx.x);
  if (row >= B) return;
  const grid_config cfg = cfgs[row];
  uint64_t h = 0;
  for (uint32_t i = 0; i < cfg.stk_depth; ++i) {
    const uint32_t sv = pool[cfg.stk_off + i];
    if (i > 0) h = node_hash(h, sv, sv < (uint32_t)tb.NS ? tb.state_sym[sv] : kNoSymbol);
    hash[cfg.stk_off + i] = h;
  }
}

bool bound(const grid_compiled* g, int which) { return g->dev[which] != nullptr || g->dev_bytes[which] == 0; }

// Raises a kernel's dynamic-LDS limit (needed above 64 KB of LDS in total)
// once per kernel, device and size.
// Raises a kernel's dynamic LDS limit once per (kernel, device, size); the
// record of what was raised is shared by all host threads.
bool raise_lds(const void* fn, uint32_t bytes) {
  struct Entry {
    const void* fn;
    int dev;
    uint32_t bytes;
  };
  static std::mutex mu;
  static Entry done[64];
  static int n_done = 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  std::lock_guard<std::mutex> lock(mu);
  for (int i = 0; i < n_done; ++i)
    if (done[i].fn == fn && done[i].dev == dev && done[i].bytes >= bytes) return true;
  if (hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) != hipSuccess) return false;
  if (n_done < 64) done[n_done++] = {fn, dev, bytes};
  return true;
}

// Resident residue workgroups on the current device (compute units x
// occupancy) for an LDS size; raises the kernel's LDS limit first.
template <int MW>
int residue_grid_size(uint32_t lds) {
  if (!raise_lds((const void*)residue_kernel<MW>, lds)) return -1;
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -1;
  // the answer per (device, LDS size), looked up once: the occupancy query
  // costs more host time than a small batch's whole mask on the device
  struct Entry {
    int dev;
    uint32_t lds;
    int blocks;
  };
  static std::mutex mu;
  static Entry seen[64];
  static int n_seen = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    for (int i = 0; i < n_seen; ++i)
      if (seen[i].dev == dev && seen[i].lds == lds) return seen[i].blocks;
  }
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, residue_kernel<MW>, kWalkThreads, lds) != hipSuccess ||
      per_cu <= 0)
    per_cu = 1;
  std::lock_guard<std::mutex> lock(mu);
  if (n_seen < 64) seen[n_seen++] = {dev, lds, cus * per_cu};
  return cus * per_cu;
}

template <int MW>
int launch_mask(const Tables& tb, int B, const grid_config* cfg_dev, const uint16_t* pool, uint32_t* mask,
                uint8_t* eos, int32_t* status, uint8_t* ws, size_t rb, uint32_t phases, hipStream_t s) {
  const uint32_t parse_bytes = prologue_lds(tb).total;
  if (!raise_lds((const void*)prologue_kernel<MW>, parse_bytes))
    return fail(GRID_E_HIP, "grid_mask: cannot raise the LDS limit");
  if (phases & GRID_PHASE_PROLOGUE) {
    hipLaunchKernelGGL(prologue_kernel<MW>, dim3(B), dim3(kProThreads), parse_bytes, s, tb, cfg_dev, pool, mask, eos,
                       ws, rb);
    const uint32_t vy = ((uint32_t)tb.max_classes + kBlock - 1) / kBlock;
    hipLaunchKernelGGL(verdict_kernel<MW>, dim3(B, vy), dim3(kBlock), verdict_lds(tb).total, s, tb, ws, rb);
  }
  if (phases & GRID_PHASE_WALK) {
    const long long blocks = 8ll * B * stream_groups(tb.V);
    if (blocks > 0x7FFFFFFFll) return fail(GRID_E_CAPACITY, "grid_mask: batch x vocabulary too large");
    hipLaunchKernelGGL(stream_kernel, dim3((uint32_t)blocks), dim3(kBlock), 0, s, tb, mask, ws, rb, B);
  }
  if ((phases & GRID_PHASE_RESIDUE) && tb.U > 0) {
    const ResLds RL = res_lds(tb, MW, B);
    const int resident = residue_grid_size<MW>(RL.total);
    if (resident <= 0) return fail(GRID_E_HIP, "grid_mask: cannot raise the residue walk's LDS limit");
    // no more workgroups than work items (a small vocabulary has few)
    const long long items = 2ll * std::min(B, RL.group) * ((tb.U + 63) / 64);
    const int blocks = (int)std::max(1ll, std::min((long long)resident, items));
    hipLaunchKernelGGL(residue_kernel<MW>, dim3(blocks), dim3(kWalkThreads), RL.total, s, tb, pool, mask, ws, rb, B);
  }
  if (phases & GRID_PHASE_FINALIZE) {
    hipLaunchKernelGGL(finalize_kernel<MW>, dim3(B), dim3(kBlock), 0, s, tb, cfg_dev, pool, mask, ws, rb, status);
    if (tb.cache && (tb.cache_flags & GRID_CACHE_INSERT))
      hipLaunchKernelGGL(cache_publish_kernel, dim3(B), dim3(kBlock), 0, s, tb, mask, ws, rb);

  }
  return GRID_OK;
}

}  // namespace

int grid::overlay_capacity() { return kFastLane; }

// head, then B rows
static size_t row_bytes(const grid_compiled* g) {
  return row_layout(g->parser.T, g->dfa.S, (int)g->vocab.spell_off.size() - 1, (int)g->classes.max_classes).total;
}

static size_t workspace_size(const grid_compiled* g, int B) { return kWsHead + row_bytes(g) * (size_t)B; }

extern "C" size_t grid_mask_workspace_bytes(const grid_compiled* g, int32_t B) {
  if (!g || B <= 0) return 0;
  return workspace_size(g, B);
}

// The device tables of a compiled handle (every artifact bound, else
// GRID_E_UNBOUND).
static int bind_tables(const grid_compiled* g, Tables& tb) {
  static const int needed[] = {GRID_ART_DFA_CLASS,   GRID_ART_BYTE_CLASS,  GRID_ART_DFA_ACCEPT_OFF,
                               GRID_ART_DFA_ACCEPT_LIST, GRID_ART_DFA_LIVE, GRID_ART_ACTION,
                               GRID_ART_PROD,        GRID_ART_TERM_INFO,   GRID_ART_SPELL_OFF,
                               GRID_ART_SPELL_BYTES, GRID_ART_SPELL_REC,   GRID_ART_SPELL_TAIL,
                               GRID_ART_ALIAS_OFF,   GRID_ART_ALIAS_IDS,   GRID_ART_LEX_FLAGS,
                               GRID_ART_LEX_HASH,    GRID_ART_LEX_SLOTS,   GRID_ART_PARSE_STATE,
                               GRID_ART_PARSE_REDX,  GRID_ART_GOTO_HASH,   GRID_ART_LEX_PREFIX,
                               GRID_ART_SPELL_OF_ID, GRID_ART_CLASS_MAP, GRID_ART_CLASS_OFF,
                               GRID_ART_CLASS_REC,   GRID_ART_LEX_STRIDE,  GRID_ART_LEX_TOKEN,
                               GRID_ART_PARSE_SHIFT, GRID_ART_GOTO_SKIP,
                               GRID_ART_STATE_SYMBOL, GRID_ART_LEX_CHILD, GRID_ART_ID_HEAD,
                               GRID_ART_LEX_TOKSUM};
  for (int w : needed)
    if (!bound(g, w)) return fail(GRID_E_UNBOUND, "artifact " + std::to_string(w) + " is not bound");
  tb.dfa = (const uint16_t*)g->dev[GRID_ART_DFA_CLASS];
  tb.bclass = (const uint8_t*)g->dev[GRID_ART_BYTE_CLASS];
  tb.acc_off = (const uint32_t*)g->dev[GRID_ART_DFA_ACCEPT_OFF];
  tb.acc_list = (const uint8_t*)g->dev[GRID_ART_DFA_ACCEPT_LIST];
  tb.live = (const uint32_t*)g->dev[GRID_ART_DFA_LIVE];
  tb.action = (const uint16_t*)g->dev[GRID_ART_ACTION];
  tb.term_info = (const uint32_t*)g->dev[GRID_ART_TERM_INFO];
  tb.pstate = (const uint32_t*)g->dev[GRID_ART_PARSE_STATE];
  tb.predx = (const uint32_t*)g->dev[GRID_ART_PARSE_REDX];
  tb.pshift = (const uint16_t*)g->dev[GRID_ART_PARSE_SHIFT];
  tb.go = (const uint16_t*)g->dev[GRID_ART_GOTO_SKIP];
  tb.ghash = (const uint2*)g->dev[GRID_ART_GOTO_HASH];
  tb.spell_off = (const uint32_t*)g->dev[GRID_ART_SPELL_OFF];
  tb.spell_bytes = (const uint8_t*)g->dev[GRID_ART_SPELL_BYTES];
  tb.spell_rec = (const uint4*)g->dev[GRID_ART_SPELL_REC];
  tb.spell_tail = (const uint4*)g->dev[GRID_ART_SPELL_TAIL];
  tb.alias_off = (const uint32_t*)g->dev[GRID_ART_ALIAS_OFF];
  tb.alias_ids = (const int32_t*)g->dev[GRID_ART_ALIAS_IDS];
  tb.lex_flags = (const uint16_t*)g->dev[GRID_ART_LEX_FLAGS];
  tb.lex_hash = (const uint32_t*)g->dev[GRID_ART_LEX_HASH];
  tb.lex_slots = (const uint32_t*)g->dev[GRID_ART_LEX_SLOTS];
  tb.lex_prefix = (const uint4*)g->dev[GRID_ART_LEX_PREFIX];
  tb.lex_stride = (const uint4*)g->dev[GRID_ART_LEX_STRIDE];
  tb.lex_token = (const uint32_t*)g->dev[GRID_ART_LEX_TOKEN];
  tb.id_head = (const uint32_t*)g->dev[GRID_ART_ID_HEAD];
  tb.lex_toksum = (const uint8_t*)g->dev[GRID_ART_LEX_TOKSUM];
  tb.lex_child = (const uint32_t*)g->dev[GRID_ART_LEX_CHILD];
  tb.spell_of_id = (const uint32_t*)g->dev[GRID_ART_SPELL_OF_ID];
  tb.state_sym = (const uint32_t*)g->dev[GRID_ART_STATE_SYMBOL];
  tb.stack_hash = nullptr;
  tb.cmap = (const uint16_t*)g->dev[GRID_ART_CLASS_MAP];
  tb.coff = (const uint32_t*)g->dev[GRID_ART_CLASS_OFF];
  tb.crec = (const uint4*)g->dev[GRID_ART_CLASS_REC];
  tb.max_classes = (int)g->classes.max_classes;
  tb.S = g->dfa.S;
  tb.C = g->dfa.C;
  tb.T = g->parser.T;
  tb.N = g->parser.N;
  tb.NS = g->parser.n_states;
  tb.P = (int)g->parser.prod.size();
  tb.U = (int)g->vocab.spell_off.size() - 1;
  tb.V = g->vocab.V;
  tb.W = (g->vocab.V + 31) / 32;
  tb.n_slots = g->lex.n_slots;
  tb.eos_id = g->vocab.eos_id;
  tb.tw = g->parser.tw;
  tb.n_pstate = (int)g->parser.pstate.size();
  tb.n_predx = (int)g->parser.predx.size();
  tb.n_pshift = (int)g->parser.pshift.size();
  tb.n_acc = (int)g->dfa.accept_list.size();
  tb.hbits = g->parser.goto_hbits;
  for (int w = 0; w < 8; ++w) tb.ign[w] = 0;
  for (int t = 0; t < tb.T && t < 256; ++t)
    if (g->term_info[t] & 1u) tb.ign[t >> 5] |= 1u << (t & 31);
  return GRID_OK;
}

static int mask_call(const grid_compiled* g, int32_t B, const grid_config* cfg_dev, const uint16_t* stack_pool_dev,
                     uint32_t* mask_dev, uint8_t* eos_dev, int32_t* status_dev, void* workspace_dev,
                     size_t workspace_bytes, void* cache_dev, size_t cache_bytes, uint32_t cache_flags,
                     uint32_t phases, void* stream, const uint64_t* stack_hash_dev = nullptr,
                     void* ci_dev = nullptr, size_t ci_bytes = 0, uint32_t ci_flags = 0) {
  clear_error();
  if (phases & ~GRID_PHASE_ALL) return fail(GRID_E_ARG, "grid_mask: unknown phase bits");
  if (cache_flags & ~(GRID_CACHE_LOOKUP | GRID_CACHE_INSERT)) return fail(GRID_E_ARG, "grid_mask: unknown cache flags");
  if (ci_flags & ~(GRID_CI_LOOKUP | GRID_CI_INSERT | GRID_CI_FAMILY | GRID_CI_GENN))
    return fail(GRID_E_ARG, "grid_mask_warm: unknown flags");
  if ((ci_flags & GRID_CI_GENN) && !(ci_flags & GRID_CI_FAMILY))
    return fail(GRID_E_ARG, "grid_mask_warm: the genN normal form belongs to the cross-family tier");
  if (!g || B <= 0 || B > 65535 || !cfg_dev || !stack_pool_dev || !mask_dev || !workspace_dev)
    return fail(GRID_E_ARG, "grid_mask: null pointer or batch size out of range");
  const size_t rb = row_bytes(g);
  if (workspace_bytes < workspace_size(g, B)) return fail(GRID_E_ARG, "grid_mask: workspace too small");
  if (((uintptr_t)workspace_dev & 255) != 0) return fail(GRID_E_ARG, "grid_mask: workspace not 256-byte aligned");
  Tables tb;
  const int brc = bind_tables(g, tb);
  if (brc != GRID_OK) return brc;
  tb.cache = nullptr;
  tb.cache_mask = 0;
  tb.cache_flags = 0;
  tb.cache_stride = cache_stride_of(tb.W);
  tb.fp = g->fingerprint;
  if (cache_dev && cache_flags) {
    const size_t n = cache_bytes / tb.cache_stride;
    if (n == 0 || (n & (n - 1)) != 0 || n > 0x80000000ull || n * tb.cache_stride != cache_bytes)
      return fail(GRID_E_ARG, "grid_mask: cache size is not grid_cache_bytes of a power of two");
    if (((uintptr_t)cache_dev & 15) != 0) return fail(GRID_E_ARG, "grid_mask: cache not 16-byte aligned");
    tb.cache = (uint8_t*)cache_dev;
    tb.cache_mask = (uint32_t)(n - 1);
    tb.cache_flags = cache_flags;
    tb.stack_hash = stack_hash_dev;
  }
  tb.ci_cache = nullptr;
  tb.ci_mask = 0;
  tb.ci_flags = 0;
  tb.ci_stride = ci_stride_of(tb.W);
  tb.family_fp = g->family_fp;
  if (ci_dev && (ci_flags & (GRID_CI_LOOKUP | GRID_CI_INSERT))) {
    const size_t n = ci_bytes / tb.ci_stride;
    if (n == 0 || (n & (n - 1)) != 0 || n > 0x80000000ull || n * tb.ci_stride != ci_bytes)
      return fail(GRID_E_ARG, "grid_mask_warm: cache size is not grid_ci_cache_bytes of a power of two");
    if (((uintptr_t)ci_dev & 15) != 0) return fail(GRID_E_ARG, "grid_mask_warm: cache not 16-byte aligned");
    tb.ci_cache = (uint8_t*)ci_dev;
    tb.ci_mask = (uint32_t)(n - 1);
    tb.ci_flags = ci_flags;
  }
  const int mw = tb.tw;
  const ResLds WL = res_lds(tb, mw, B);
  if (tb.T > 255 || (mw != 2 && mw != 4 && mw != 8) || WL.total + 64 > kWalkLdsMax ||
      prologue_parse_lds(tb).total > kPrologueParseMax || verdict_lds(tb).total > 64 * 1024)
    return fail(GRID_E_CAPACITY, "grid_mask: lexer DFA or LR tables too large for the LDS staging");
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace_dev;
  int rc;
  if (mw == 2)
    rc = launch_mask<2>(tb, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, ws, rb, phases, s);
  else if (mw == 4)
    rc = launch_mask<4>(tb, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, ws, rb, phases, s);
  else
    rc = launch_mask<8>(tb, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, ws, rb, phases, s);
  if (rc != GRID_OK) return rc;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_mask launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

extern "C" int grid_mask_phases(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                                const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                                int32_t* status_dev, void* workspace_dev, size_t workspace_bytes,
                                uint32_t phases, void* stream) {
  return mask_call(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, workspace_dev, workspace_bytes,
                   nullptr, 0, 0, phases, stream);
}

extern "C" int grid_mask(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                         const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                         int32_t* status_dev, void* workspace_dev, size_t workspace_bytes, void* stream) {
  return mask_call(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, workspace_dev, workspace_bytes,
                   nullptr, 0, 0, GRID_PHASE_ALL, stream);
}

extern "C" int grid_mask_cached(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                                const uint16_t* stack_pool_dev, const uint64_t* stack_hash_dev, uint32_t* mask_dev,
                                uint8_t* eos_dev, int32_t* status_dev, void* workspace_dev, size_t workspace_bytes,
                                void* cache_dev, size_t cache_bytes, uint32_t cache_flags, void* stream) {
  return mask_call(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, workspace_dev, workspace_bytes,
                   cache_dev, cache_bytes, cache_flags, GRID_PHASE_ALL, stream, stack_hash_dev);
}

extern "C" int grid_stack_hash(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                               const uint16_t* stack_pool_dev, uint64_t* stack_hash_dev, void* stream) {
  clear_error();
  if (!g || B <= 0 || !cfg_dev || !stack_pool_dev || !stack_hash_dev)
    return fail(GRID_E_ARG, "grid_stack_hash: null pointer or bad batch size");
  Tables tb;
  const int rc = bind_tables(g, tb);
  if (rc != GRID_OK) return rc;
  hipLaunchKernelGGL(stack_hash_kernel, dim3((unsigned)((B + 63) / 64)), dim3(64), 0, (hipStream_t)stream, tb, cfg_dev,
                     stack_pool_dev, stack_hash_dev, B);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_stack_hash launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

// ------------------------------------------------------ no-alloc mask entry
// The workspace of grid_mask_noalloc: a device array of the code object, one
// copy per GPU, held until the process ends.  Host code never passes the
// array's name to a kernel (on the host it is only a stand-in for the
// symbol); it uses the device address hipGetSymbolAddress returns, looked up
// once per device with that device current.
constexpr size_t kScratchBytes = size_t(32) << 20;
static __device__ __align__(256) uint8_t scratch[kScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's scratch array, or nullptr (the
// error is recorded).
void* scratch_on_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    fail(GRID_E_HIP, "grid_mask_noalloc: no current device");
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      fail(GRID_E_HIP, std::string("grid_mask_noalloc: hipGetSymbolAddress: ") + hipGetErrorString(e));
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}
}  // namespace

extern "C" size_t grid_mask_noalloc_max_bytes(void) { return kScratchBytes; }

extern "C" int grid_mask_noalloc(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                                 const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                                 int32_t* status_dev, void* stream) {
  clear_error();
  if (!g || B <= 0 || B > 65535) return fail(GRID_E_ARG, "grid_mask_noalloc: null handle or batch size out of range");
  const size_t need = workspace_size(g, B);
  if (need > kScratchBytes)
    return fail(GRID_E_CAPACITY, "grid_mask_noalloc: " + std::to_string(B) + " rows need " + std::to_string(need) +
                                     " workspace bytes, more than the " + std::to_string(kScratchBytes) +
                                     " of the static scratch array");
  void* ws = scratch_on_current_device();
  if (!ws) return GRID_E_HIP;
  return mask_call(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, ws, kScratchBytes, nullptr, 0, 0,
                   GRID_PHASE_ALL, stream);
}

extern "C" size_t grid_cache_bytes(const grid_compiled* g, int32_t n_entries) {
  if (!g || n_entries < 1 || (n_entries & (n_entries - 1)) != 0) return 0;
  return (size_t)n_entries * cache_stride_of((g->vocab.V + 31) / 32);
}

extern "C" int grid_cache_clear(const grid_compiled* g, void* cache_dev, size_t cache_bytes, void* stream) {
  clear_error();
  if (!g || !cache_dev) return fail(GRID_E_ARG, "grid_cache_clear: null argument");
  const uint32_t stride = cache_stride_of((g->vocab.V + 31) / 32);
  const size_t n = cache_bytes / stride;
  if (n == 0 || (n & (n - 1)) != 0 || n > 0x80000000ull || n * stride != cache_bytes)
    return fail(GRID_E_ARG, "grid_cache_clear: cache size is not grid_cache_bytes of a power of two");
  const int blocks = (int)std::min<size_t>((n + kBlock - 1) / kBlock, 1024);
  hipLaunchKernelGGL(cache_clear_kernel, dim3(blocks), dim3(kBlock), 0, (hipStream_t)stream, (uint8_t*)cache_dev,
                     (uint32_t)n, stride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_cache_clear launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

static int accept_call(const grid_compiled* g, int32_t B, const grid_config* cfg_dev, const uint16_t* stack_pool_dev,
                       const int32_t* token_dev, grid_config* cfg_out_dev, uint16_t* stack_out_dev, uint64_t* hash_dev,
                       uint32_t stack_cap, int32_t* status_dev, int inplace, void* stream, int tok_stride = 1) {
  Tables tb;
  const int rc = bind_tables(g, tb);
  if (rc != GRID_OK) return rc;
  if (tb.T > 255) return fail(GRID_E_CAPACITY, "grid_accept: more than 255 terminals");
  const ParseLds PL = prologue_parse_lds(tb);
  const int use_lds = PL.total <= kPrologueParseMax ? 1 : 0;
  uint32_t lds = use_lds ? PL.total + pad16(accept_stack_cap(stack_cap) * 2u) : 0u;
  const int use_lex = use_lds && lds + accept_lex_lds(tb).total <= kAcceptLdsMax ? 1 : 0;
  if (use_lex) lds += accept_lex_lds(tb).total;
  const void* fn = tb.tw == 2 ? (const void*)accept_kernel<2>
                              : (tb.tw == 4 ? (const void*)accept_kernel<4> : (const void*)accept_kernel<8>);
  if (!raise_lds(fn, lds)) return fail(GRID_E_HIP, "grid_accept: cannot raise the LDS limit");
  hipStream_t s = (hipStream_t)stream;
  const dim3 grid((unsigned)B), block(kBlock);
  if (tb.tw == 2)
    hipLaunchKernelGGL(accept_kernel<2>, grid, block, lds, s, tb, cfg_dev, stack_pool_dev, token_dev, cfg_out_dev,
                       stack_out_dev, hash_dev, stack_cap, status_dev, use_lds, use_lex, inplace, tok_stride);
  else if (tb.tw == 4)
    hipLaunchKernelGGL(accept_kernel<4>, grid, block, lds, s, tb, cfg_dev, stack_pool_dev, token_dev, cfg_out_dev,
                       stack_out_dev, hash_dev, stack_cap, status_dev, use_lds, use_lex, inplace, tok_stride);
  else
    hipLaunchKernelGGL(accept_kernel<8>, grid, block, lds, s, tb, cfg_dev, stack_pool_dev, token_dev, cfg_out_dev,
                       stack_out_dev, hash_dev, stack_cap, status_dev, use_lds, use_lex, inplace, tok_stride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_accept launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

extern "C" size_t grid_ci_cache_bytes(const grid_compiled* g, int32_t n_entries) {
  if (!g || n_entries < 1 || (n_entries & (n_entries - 1)) != 0) return 0;
  return (size_t)n_entries * ci_stride_of((g->vocab.V + 31) / 32);
}

extern "C" int grid_ci_cache_clear(const grid_compiled* g, void* cache_dev, size_t cache_bytes, void* stream) {
  clear_error();
  if (!g || !cache_dev) return fail(GRID_E_ARG, "grid_ci_cache_clear: null argument");
  const uint32_t stride = ci_stride_of((g->vocab.V + 31) / 32);
  const size_t n = cache_bytes / stride;
  if (n == 0 || (n & (n - 1)) != 0 || n > 0x80000000ull || n * stride != cache_bytes)
    return fail(GRID_E_ARG, "grid_ci_cache_clear: cache size is not grid_ci_cache_bytes of a power of two");
  const int blocks = (int)std::min<size_t>((n + kBlock - 1) / kBlock, 1024);
  hipLaunchKernelGGL(cache_clear_kernel, dim3(blocks), dim3(kBlock), 0, (hipStream_t)stream, (uint8_t*)cache_dev,
                     (uint32_t)n, stride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_ci_cache_clear launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

extern "C" int grid_mask_warm(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                              const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev, int32_t* status_dev,
                              void* workspace_dev, size_t workspace_bytes, void* ci_cache_dev, size_t ci_cache_bytes,
                              uint32_t ci_flags, void* stream) {
  return mask_call(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, workspace_dev, workspace_bytes,
                   nullptr, 0, 0, GRID_PHASE_ALL, stream, nullptr, ci_cache_dev, ci_cache_bytes, ci_flags);
}

extern "C" int grid_accept(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                           const uint16_t* stack_pool_dev, const int32_t* token_dev, grid_config* cfg_out_dev,
                           uint16_t* stack_out_dev, uint32_t stack_cap, int32_t* status_dev, void* stream) {
  clear_error();
  if (!g || B <= 0 || !cfg_dev || !stack_pool_dev || !token_dev || !cfg_out_dev || !stack_out_dev || stack_cap < 2)
    return fail(GRID_E_ARG, "grid_accept: null pointer or bad size");
  return accept_call(g, B, cfg_dev, stack_pool_dev, token_dev, cfg_out_dev, stack_out_dev, nullptr, stack_cap,
                     status_dev, 0, stream);
}

extern "C" int grid_accept_inplace(const grid_compiled* g, int32_t B, grid_config* cfg_dev, uint16_t* stack_pool_dev,
                                   uint64_t* stack_hash_dev, uint32_t stack_cap, const int32_t* token_dev,
                                   int32_t* status_dev, void* stream) {
  clear_error();
  if (!g || B <= 0 || !cfg_dev || !stack_pool_dev || !token_dev || stack_cap < 2)
    return fail(GRID_E_ARG, "grid_accept_inplace: null pointer or bad size");
  return accept_call(g, B, cfg_dev, stack_pool_dev, token_dev, cfg_dev, stack_pool_dev, stack_hash_dev, stack_cap,
                     status_dev, 1, stream);
}

// Jump-forward step i (section 6.1 step 6): a row whose mask allows exactly
// one token (the end-of-sequence token counts when its bit is set) takes it
// as span[row][i]; any other row, a row whose mask call did not end OK, and a
// row whose span already stopped (a non-forced step, or the end-of-sequence
// token) gets -1.  Before that, a row whose advance by span[row][i - 1]
// failed (acc_status neither OK nor FINISHED; its configuration is then
// unchanged) has that token taken back and stops.  span_len[row] counts the
// forced tokens.  With take == 0 only the check of the last advance runs.
__global__ __launch_bounds__(kBlock) void singleton_kernel(const uint32_t* __restrict__ mask,
                                                           const int32_t* __restrict__ status,
                                                           const int32_t* __restrict__ acc_status, int32_t* span,
                                                           int32_t* span_len, int W, int max_len, int i, int eos_id,
                                                           int take) {
  const int row = (int)blockIdx.x, tid = (int)threadIdx.x;
  __shared__ int count, word;
  if (tid == 0) {
    count = 0;
    word = -1;
  }
  __syncthreads();
  const uint32_t* m = mask + (size_t)row * W;
  int c = 0, wd = -1;
  if (take) {
    for (int w = tid; w < W; w += kBlock) {
      const int k = __popc(m[w]);
      c += k;
      if (k) wd = w;
    }
  }
  if (c) atomicAdd(&count, c);
  if (wd >= 0) atomicMax(&word, wd);
  __syncthreads();
  if (tid != 0) return;
  int32_t* sp = span + (size_t)row * max_len;
  if (i == 0) span_len[row] = 0;
  bool open = i == 0 || (sp[i - 1] >= 0 && sp[i - 1] != eos_id);
  if (i > 0 && sp[i - 1] >= 0 && acc_status[row] != GRID_ROW_OK && acc_status[row] != GRID_ROW_FINISHED) {
    sp[i - 1] = -1;  // not applied: the row keeps the configuration before it
    span_len[row] = i - 1;
    open = false;
  }
  if (!take) return;
  int tok = -1;
  if (open && count == 1 && (!status || status[row] == GRID_ROW_OK)) tok = word * 32 + __ffs((int)m[word]) - 1;
  sp[i] = tok;
  if (tok >= 0) span_len[row] = i + 1;
}

extern "C" int grid_forced_span(const grid_compiled* g, int32_t B, grid_config* cfg_dev, uint16_t* stack_pool_dev,
                                uint64_t* stack_hash_dev, uint32_t stack_cap, int32_t max_len, int32_t* span_dev,
                                int32_t* span_len_dev, uint32_t* mask_dev, uint8_t* eos_dev, int32_t* status_dev,
                                void* workspace_dev, size_t workspace_bytes, void* stream) {
  clear_error();
  if (!g || B <= 0 || !cfg_dev || !stack_pool_dev || !span_dev || !span_len_dev || !mask_dev || !status_dev ||
      !workspace_dev || max_len < 1 || stack_cap < 2)
    return fail(GRID_E_ARG, "grid_forced_span: null pointer or bad size");
  const size_t mask_ws = workspace_size(g, B);
  if (workspace_bytes < mask_ws + (size_t)B * 4u)
    return fail(GRID_E_ARG, "grid_forced_span: workspace smaller than grid_forced_span_workspace_bytes");
  // the advances' statuses live after the mask workspace
  int32_t* acc_status = (int32_t*)((uint8_t*)workspace_dev + mask_ws);
  const int W = (g->vocab.V + 31) / 32;
  hipStream_t s = (hipStream_t)stream;
  for (int i = 0; i <= max_len; ++i) {
    int rc = mask_call(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, workspace_dev, mask_ws, nullptr,
                       0, 0, GRID_PHASE_ALL, stream);
    if (rc != GRID_OK) return rc;
    const int take = i < max_len ? 1 : 0;  // the last round only checks the last advance
    hipLaunchKernelGGL(singleton_kernel, dim3((unsigned)B), dim3(kBlock), 0, s, mask_dev, status_dev, acc_status,
                       span_dev, span_len_dev, W, max_len, i, g->vocab.eos_id, take);
    if (!take) break;
    // rows with -1 are left as they are (their status is not needed)
    rc = accept_call(g, B, cfg_dev, stack_pool_dev, span_dev + i, cfg_dev, stack_pool_dev, stack_hash_dev, stack_cap,
                     acc_status, 1, stream, max_len);
    if (rc != GRID_OK) return rc;
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_forced_span launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

extern "C" size_t grid_forced_span_workspace_bytes(const grid_compiled* g, int32_t B) {
  if (!g || B <= 0) return 0;
  return workspace_size(g, B) + (size_t)B * 4u;
}

extern "C" int grid_apply(const uint32_t* mask_dev, void* logits_dev, int32_t dtype, int32_t B, int32_t V,
                          int64_t row_stride, void* stream) {
  clear_error();
  if (!mask_dev || !logits_dev || B <= 0 || V <= 0 || row_stride < V)
    return fail(GRID_E_ARG, "grid_apply: null pointer or bad shape");
  if (dtype != GRID_DTYPE_F32 && dtype != GRID_DTYPE_BF16) return fail(GRID_E_ARG, "grid_apply: dtype");
  const int W = (V + 31) / 32;
  if (B > 65535) return fail(GRID_E_ARG, "grid_apply: more than 65535 rows");
  const int groups = (V + 7) / 8;
  // one grid row per batch row; along it enough workgroups for every group
  // of 8 logits, at most 512 (a grid-stride loop covers the rest)
  const dim3 blocks((unsigned)std::min((groups + kBlock - 1) / kBlock, 512), (unsigned)B);
  hipStream_t s = (hipStream_t)stream;
  const size_t esz = dtype == GRID_DTYPE_BF16 ? 2 : 4;
  const bool vec_ok = ((uintptr_t)logits_dev % 16 == 0) && ((row_stride * (int64_t)esz) % 16 == 0);
  if (dtype == GRID_DTYPE_BF16)
    hipLaunchKernelGGL(apply_kernel<uint16_t>, blocks, dim3(kBlock), 0, s, mask_dev,
                       (uint16_t*)logits_dev, B, V, W, row_stride, 0xFF80u, vec_ok);
  else
    hipLaunchKernelGGL(apply_kernel<uint32_t>, blocks, dim3(kBlock), 0, s, mask_dev,
                       (uint32_t*)logits_dev, B, V, W, row_stride, 0xFF800000u, vec_ok);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_apply launch: ") + hipGetErrorString(e));
  return GRID_OK;
}
