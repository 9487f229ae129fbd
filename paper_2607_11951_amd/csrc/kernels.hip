// kernels.hip -- device side of the cold exact mask and the -inf apply (gfx950).
//
// grid_mask launches, on the caller's stream:
//  1. prologue (8 workgroups per row): every workgroup stages the compact LR
//     tables and the top of the row's stack in LDS and computes the allowed
//     terminals A(sigma) (section 3.2, allowed terminals under table
//     compression) by simulating the reduce chain for the whole set of
//     terminals at once: at each state the terminals that shift are allowed,
//     those reduced by the state's production travel on together, the rest
//     are errors.  Each workgroup then records, for its share of the allowed
//     terminals, the stack after that terminal's shift (on a private overlay
//     above the shared read-only stack), that stack's own allowed set, and the
//     trailing-lexeme codes of every lexer state under it.  Workgroup 0 also
//     resolves the pending lexeme (its winner at an emission), the end-of-
//     sequence gate (section 3.2, EOS gating, mid-lexeme aware), the trailing
//     codes under A(sigma) (Definition 2), and a 256-entry first-byte table:
//     the scan state after any first byte of a token (continuing the pending
//     lexeme, or emitting it and starting a new one), or "rejected"; it clears
//     the row's mask words.
//  2. walk (persistent; work items = row x spelling tile): one lane per
//     distinct spelling in byte order, so neighbouring lanes share prefixes
//     and die together.  The lexer DFA, compact LR tables, byte classes,
//     accept lists, first-byte table and trailing codes sit in LDS; each
//     spelling's first 8 bytes and first alias id arrive in one 16-byte load.
//     A byte that kills the DFA emits the pending lexeme as the highest-
//     priority candidate that is allowed (or ignored) and passes the schema
//     lexicon, then the byte is scanned again (section 4.1, trie walk).
//     Tokens that stay in one lexeme are decided by the trailing codes
//     (context-independent part, section 4.2); after one shift the recorded
//     stack, allowed set and codes are used; later shifts run reduce chains on
//     the lane's own LDS overlay (context-dependent part, Proposition 4).
//     Rejection is monotone, so a lane stops at its first failing byte.
//     Allowed spellings set the bits of every alias id; a lane whose LDS stack
//     area is too small hands its spelling to the slow path.
//  3. finalize (one workgroup per row): re-walks handed-over spellings with a
//     large stack area in the workspace, writes the row status and flags an
//     empty mask (Proposition 8: a viable configuration has a nonempty mask).
// grid_apply is a streaming in-place -inf fill of the masked logits.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <string>

#include "host.h"
#include "lexhash.h"

namespace grid {
int fail(int code, const std::string& msg);
void clear_error();
}  // namespace grid

using namespace grid;

namespace {

constexpr int kBlock = 256;          // prologue / apply workgroup size
constexpr int kProGroups = 8;        // prologue workgroups per row
constexpr int kStackWin = 256;       // top of the row's stack kept in LDS (prologue)
constexpr int kPostCap = 14;         // overlay states recorded per first shift
constexpr int kTmpCap = 32;          // prologue: virtual pushes of one simulation
constexpr int kGuard = 4096;         // reduce-chain step bound
constexpr int kAccCap = 4096;        // accept-list bytes staged in LDS by the walk
constexpr int kSlowCap = 4096;       // spellings handed to the slow path per row
constexpr int kSlowThreads = 64;
constexpr int kSlowLane = 512;       // slow path per-thread stack area (workspace)
constexpr uint32_t kRowValid = 0x600D;
constexpr size_t kWsHead = 256;      // workspace head: the walk's work counter
constexpr int kMaxRounds = 257;      // set-simulation reruns (each peels one reduce group)

// walk launch shape
constexpr int kWalkThreads = 512;
constexpr int kWalkSpt = 2;          // spellings per thread
constexpr int kWalkTile = kWalkThreads * kWalkSpt;
constexpr int kFastLane = 16;        // per-lane stack area in LDS (overlay at the bottom,
                                     // virtual pushes above it)

struct Tables {
  const uint16_t* dfa;        // [S*C]
  const uint8_t* bclass;      // [256]
  const uint32_t* acc_off;    // [S+1]
  const uint8_t* acc_list;
  const uint32_t* live;       // [S*8]
  const uint16_t* action;     // [NS*(T+1)] (shift targets)
  const uint32_t* prod;       // [P]
  const uint32_t* term_info;  // [T]
  const uint32_t* pstate;     // [NS][2*tw+2]
  const uint32_t* predx;
  const uint32_t* goff;       // [NS+1]
  const uint32_t* gent;
  const uint32_t* spell_off;  // [U+1]
  const uint8_t* spell_bytes;
  const uint4* spell_rec;     // [U]: head lo, head hi, first id | multi << 31, length
  const uint32_t* alias_off;  // [U+1]
  const int32_t* alias_ids;
  const uint16_t* lex_flags;
  const uint32_t* lex_hash;
  const uint32_t* lex_slots;
  int S, C, T, N, NS, P, U, V, W, n_slots, eos_id;
  int tw, n_pstate, n_predx, n_gent, n_acc;
};

// ---------------------------------------------------------------- workspace
struct RowHeader {
  uint32_t A[8];
  uint32_t eos_ok;
  uint32_t valid;
  int32_t winner;             // pending lexeme's winner at an emission, -1 none
  uint32_t slow_count;
  int32_t pstat[kProGroups];  // status bits from each prologue workgroup
  int32_t wstat;              // status bits from the walk
  uint32_t pad[11];
};
static_assert(sizeof(RowHeader) == 128, "row header is 128 bytes");

struct Post {                 // stack after shifting one allowed terminal
  uint16_t k;                 // shared base entries kept
  uint8_t m;                  // overlay entries
  uint8_t ok;
  uint16_t ov[kPostCap];
};
static_assert(sizeof(Post) == 32, "post entry is 32 bytes");

struct RowLayout {
  size_t post, a2, vend, fb, slow, slow_ov, vend1, total;
  size_t s_pad;  // trailing-code row stride (entries)
};

__host__ __device__ inline RowLayout row_layout(int T, int S) {
  RowLayout L;
  size_t o = sizeof(RowHeader);
  L.post = o;
  o += (size_t)T * sizeof(Post);
  L.a2 = o;
  o += (size_t)T * 32;
  L.vend = o;
  o += ((size_t)S * 2 + 15) & ~(size_t)15;
  L.fb = o;
  o += 256 * 8;
  L.slow = o;
  o += kSlowCap * 4;
  L.slow_ov = o;
  o += (size_t)kSlowThreads * kSlowLane * 2;
  L.s_pad = ((size_t)S + 7) & ~(size_t)7;
  L.vend1 = o;
  o += (size_t)T * L.s_pad * 2;
  L.total = (o + 255) & ~(size_t)255;
  return L;
}

// first-byte table entry: x = q | kind << 16 | t1 << 24 (kind 0 rejected,
// 1 alive on sigma, 2 alive after shifting t1); y = lexicon node
constexpr uint32_t kFbDead = 0, kFbMode0 = 1, kFbMode1 = 2;

__host__ __device__ inline uint32_t pad16(uint32_t x) { return (x + 15u) & ~15u; }

// Copies bytes from global to LDS with 16-byte loads (both 16-byte aligned).
__device__ inline void stage16(uint8_t* dst, const uint8_t* src, uint32_t bytes, int tid, int nt) {
  const uint32_t n16 = bytes >> 4;
#pragma unroll 4
  for (uint32_t i = tid; i < n16; i += nt) reinterpret_cast<uint4*>(dst)[i] = reinterpret_cast<const uint4*>(src)[i];
  for (uint32_t i = (n16 << 4) + tid; i < bytes; i += nt) dst[i] = src[i];
}

// ------------------------------------------------------- compact LR tables
struct ParseTabs {  // pointers into LDS (or global memory)
  const uint32_t* st;
  const uint32_t* redx;
  const uint32_t* goff;
  const uint32_t* gent;
  const uint32_t* prod;
  const uint16_t* action;  // global, dense: shift targets
  int tw, stride, T;
};

struct ParseLds {  // byte offsets of the staged tables
  uint32_t st, redx, goff, gent, prod, total;
};

__host__ __device__ inline ParseLds parse_lds(const Tables& tb, uint32_t base) {
  ParseLds L;
  uint32_t o = base;
  L.st = o;
  o += pad16((uint32_t)tb.n_pstate * 4);
  L.redx = o;
  o += pad16((uint32_t)tb.n_predx * 4);
  L.goff = o;
  o += pad16((uint32_t)(tb.NS + 1) * 4);
  L.gent = o;
  o += pad16((uint32_t)tb.n_gent * 4);
  L.prod = o;
  o += pad16((uint32_t)tb.P * 4);
  L.total = o - base;
  return L;
}

__device__ inline ParseTabs stage_parse(const Tables& tb, uint8_t* lds, const ParseLds& L, int tid, int nt) {
  stage16(lds + L.st, (const uint8_t*)tb.pstate, (uint32_t)tb.n_pstate * 4, tid, nt);
  stage16(lds + L.redx, (const uint8_t*)tb.predx, (uint32_t)tb.n_predx * 4, tid, nt);
  stage16(lds + L.goff, (const uint8_t*)tb.goff, (uint32_t)(tb.NS + 1) * 4, tid, nt);
  stage16(lds + L.gent, (const uint8_t*)tb.gent, (uint32_t)tb.n_gent * 4, tid, nt);
  stage16(lds + L.prod, (const uint8_t*)tb.prod, (uint32_t)tb.P * 4, tid, nt);
  return {(const uint32_t*)(lds + L.st),   (const uint32_t*)(lds + L.redx), (const uint32_t*)(lds + L.goff),
          (const uint32_t*)(lds + L.gent), (const uint32_t*)(lds + L.prod), tb.action,
          tb.tw,                           2 * tb.tw + 2,                    tb.T};
}

__device__ inline ParseTabs global_parse(const Tables& tb) {
  return {tb.pstate, tb.predx, tb.goff, tb.gent, tb.prod, tb.action, tb.tw, 2 * tb.tw + 2, tb.T};
}

struct BaseStack {  // the shared read-only stack of one row
  const uint16_t* pool;  // states [0, depth)
  const uint16_t* win;   // copy of states [lo, depth) (LDS), or null with lo = depth
  uint32_t depth, lo;
  __device__ uint16_t at(uint32_t i) const { return i >= lo ? win[i - lo] : pool[i]; }
};

__device__ inline uint16_t goto_of(const ParseTabs& pt, uint32_t s, uint32_t a) {
  for (uint32_t j = pt.goff[s]; j < pt.goff[s + 1]; ++j) {
    const uint32_t e = pt.gent[j];
    if ((e & 0xFFFFu) == a) return (uint16_t)(e >> 16);
  }
  return kNoGoto;
}

// Action of terminal x in state s: -2 shift (or accept for the end-of-input
// column), -1 error, else the production to reduce.
__device__ inline int action_of(const ParseTabs& pt, uint32_t s, int x) {
  const uint32_t* rec = pt.st + (size_t)s * pt.stride;
  const uint32_t w = (uint32_t)x >> 5, bit = 1u << (x & 31);
  if (rec[w] & bit) return -2;
  const uint32_t info = rec[2 * pt.tw];
  if (rec[pt.tw + w] & bit) return (int)(info & 0xFFFFu);
  const uint32_t nx = info >> 16;
  const uint32_t* g = pt.redx + rec[2 * pt.tw + 1];
  for (uint32_t e = 0; e < nx; ++e, g += pt.tw + 1)
    if (g[1 + w] & bit) return (int)g[0];
  return -1;
}

// Virtual stack base[0,k) ++ ov[0,m) ++ tmp[0,t).
#define GRID_TOP(k, m, t) ((t) > 0 ? tmp[(t)-1] : ((m) > 0 ? ov[(m)-1] : bs.at((k)-1)))

// Reduce chain of terminal x, not changing the stack.  1 shift, 2 accept (x
// is the end of input), 0 error, -1 capacity.
__device__ int sim1_test(const ParseTabs& pt, const BaseStack& bs, uint32_t k, int m, const uint16_t* ov,
                         uint16_t* tmp, int tmpcap, int x) {
  int t = 0;
  for (int guard = 0; guard < kGuard; ++guard) {
    const uint16_t s = GRID_TOP(k, m, t);
    const int a = action_of(pt, s, x);
    if (a == -2) return x == pt.T ? 2 : 1;
    if (a < 0) return 0;
    const uint32_t pr = pt.prod[a];
    uint32_t len = pr >> 16;
    uint32_t d = min((uint32_t)t, len);
    t -= (int)d;
    len -= d;
    d = min((uint32_t)m, len);
    m -= (int)d;
    len -= d;
    if (len >= k) return 0;
    k -= len;
    const uint16_t g = goto_of(pt, GRID_TOP(k, m, t), pr & 0xFFFFu);
    if (g == kNoGoto) return 0;
    if (t >= tmpcap) return -1;
    tmp[t++] = g;
  }
  return -1;
}

// Reduce chain of terminal x applied to (k, m, ov), then its shift.
__device__ int sim1_shift(const ParseTabs& pt, const BaseStack& bs, uint32_t& k, int& m, uint16_t* ov, int cap,
                          int x) {
  const uint16_t* tmp = nullptr;  // unused by GRID_TOP with t = 0
  (void)tmp;
  for (int guard = 0; guard < kGuard; ++guard) {
    const uint16_t s = m > 0 ? ov[m - 1] : bs.at(k - 1);
    const int a = action_of(pt, s, x);
    if (a == -2) {
      if (x == pt.T) return 2;
      if (m >= cap) return -1;
      ov[m++] = (uint16_t)(pt.action[(size_t)s * (pt.T + 1) + x] & 0x3FFF);
      return 1;
    }
    if (a < 0) return 0;
    const uint32_t pr = pt.prod[a];
    uint32_t len = pr >> 16;
    const uint32_t d = min((uint32_t)m, len);
    m -= (int)d;
    len -= d;
    if (len >= k) return 0;
    k -= len;
    const uint16_t under = m > 0 ? ov[m - 1] : bs.at(k - 1);
    const uint16_t g = goto_of(pt, under, pr & 0xFFFFu);
    if (g == kNoGoto) return 0;
    if (m >= cap) return -1;
    ov[m++] = g;
  }
  return -1;
}

// Set simulation: acc |= the terminals of X that can be shifted next from
// base[0,k0) ++ ov[0,m0).  All of X runs one reduce chain; at each state the
// shifting terminals are accepted, those reduced by one production continue
// together, terminals of another reduce production of the same state rerun
// from the start, the rest fail.  MW = words per set (>= tw).  0 ok, -1
// capacity (acc is then incomplete).
template <int MW>
__device__ int sim_set(const ParseTabs& pt, const BaseStack& bs, uint32_t k0, int m0, const uint16_t* ov,
                       uint16_t* tmp, int tmpcap, const uint32_t (&X)[MW], uint32_t (&acc)[MW]) {
  uint32_t todo[MW];
#pragma unroll
  for (int w = 0; w < MW; ++w) todo[w] = X[w];
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
    uint32_t k = k0;
    int m = m0, t = 0;
    for (int guard = 0; guard < kGuard; ++guard) {
      const uint16_t s = GRID_TOP(k, m, t);
      const uint32_t* rec = pt.st + (size_t)s * pt.stride;
      uint32_t nxt[MW], live = 0;
#pragma unroll
      for (int w = 0; w < MW; ++w) {
        const uint32_t sh = w < pt.tw ? rec[w] : 0u;
        const uint32_t rd = w < pt.tw ? rec[pt.tw + w] : 0u;
        acc[w] |= cur[w] & sh;
        nxt[w] = cur[w] & rd;
        live |= nxt[w];
      }
      const uint32_t info = rec[2 * pt.tw];
      int chosen = live ? (int)(info & 0xFFFFu) : -1;
      const uint32_t nx = info >> 16;
      const uint32_t* g = pt.redx + rec[2 * pt.tw + 1];
      for (uint32_t e = 0; e < nx; ++e, g += pt.tw + 1) {
        uint32_t gl = 0, part[MW];
#pragma unroll
        for (int w = 0; w < MW; ++w) {
          part[w] = cur[w] & (w < pt.tw ? g[1 + w] : 0u);
          gl |= part[w];
        }
        if (!gl) continue;
        if (chosen < 0) {
          chosen = (int)g[0];
#pragma unroll
          for (int w = 0; w < MW; ++w) nxt[w] = part[w];
        } else {
#pragma unroll
          for (int w = 0; w < MW; ++w) todo[w] |= part[w];
        }
      }
      if (chosen < 0) break;
#pragma unroll
      for (int w = 0; w < MW; ++w) cur[w] = nxt[w];
      const uint32_t pr = pt.prod[chosen];
      uint32_t len = pr >> 16;
      uint32_t d = min((uint32_t)t, len);
      t -= (int)d;
      len -= d;
      d = min((uint32_t)m, len);
      m -= (int)d;
      len -= d;
      if (len >= k) break;
      k -= len;
      const uint16_t gs = goto_of(pt, GRID_TOP(k, m, t), pr & 0xFFFFu);
      if (gs == kNoGoto) break;
      if (t >= tmpcap) return -1;
      tmp[t++] = gs;
    }
  }
  uint32_t any = 0;
#pragma unroll
  for (int w = 0; w < MW; ++w) any |= todo[w];
  return any ? -1 : 0;
}

// ---------------------------------------------------------- lexicon helpers
struct Slot {
  uint32_t fbase, hbase, hmask, restricted, nodes;
};

__device__ inline Slot load_slot(const Tables& tb, int s) {
  const uint32_t* r = tb.lex_slots + (size_t)s * kSlotWords;
  return {r[0], r[1], r[2], r[3], r[4]};
}

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

// Category c of terminal info ti restricts the lexeme in this slot.
__device__ inline bool restricted_cat(const Slot& sl, uint32_t ti, uint32_t& c) {
  c = (ti >> 8) & 0xFF;
  return c != 0xFF && ((sl.restricted >> c) & 1u);
}

// Trailing-lexeme code of DFA state q under allowed set bits8 plus the
// ignored set I8: bit 15 = viable through an unrestricted terminal, bits
// 0..7 = categories whose lexicon prefix test decides (Definition 2).
__device__ inline uint16_t state_code(const Tables& tb, const Slot& sl, int q, const uint32_t* bits8,
                                      const uint32_t* I8) {
  uint32_t code = 0;
  for (int wd = 0; wd < 8; ++wd) {
    uint32_t bits = tb.live[(size_t)q * 8 + wd] & (bits8[wd] | I8[wd]);
    while (bits) {
      const int t = wd * 32 + __ffs(bits) - 1;
      bits &= bits - 1;
      uint32_t c;
      if (restricted_cat(sl, tb.term_info[t], c)) code |= 1u << c;
      else code |= 0x8000u;
    }
  }
  return (uint16_t)code;
}

__device__ inline bool code_ok(uint32_t code, uint32_t lf) { return (code & 0x8000u) || (lf & code & 0xFFu); }

// ---------------------------------------------------------------- prologue
template <int MW>
__global__ __launch_bounds__(kBlock) void prologue_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                          const uint16_t* __restrict__ pool,
                                                          uint32_t* __restrict__ mask,
                                                          uint8_t* __restrict__ eos_out,
                                                          uint8_t* __restrict__ ws, size_t rbytes) {
  extern __shared__ __align__(16) uint8_t plds[];
  const int row = blockIdx.x;
  const int grp = blockIdx.y;
  const int tid = threadIdx.x;
  __shared__ uint16_t win[kStackWin];
  __shared__ uint32_t A[8], I[8], Aw[8], ALL[8];
  __shared__ uint32_t A2s[256 * 8];
  __shared__ Post posts[256];
  __shared__ uint16_t scratch[kBlock][kPostCap + kTmpCap];
  __shared__ uint8_t glist[256];  // allowed terminals this workgroup expands
  __shared__ int nG, bad, overflow, winner;
  if (row == 0 && grp == 0 && tid == 0) *(uint32_t*)ws = 0u;  // walk work counter
  uint8_t* rw = ws + kWsHead + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  const RowLayout L = row_layout(tb.T, tb.S);
  Post* post = (Post*)(rw + L.post);
  uint32_t* a2 = (uint32_t*)(rw + L.a2);
  const grid_config cfg = cfgs[row];
  uint32_t* mrow = mask + (size_t)row * tb.W;
  const ParseTabs pt = stage_parse(tb, plds, parse_lds(tb, 0), tid, kBlock);

  if (tid == 0) {
    int b = 0;
    if (cfg.q >= tb.S || cfg.slot >= tb.n_slots || cfg.stk_depth < 1) b = 1;
    if (!b) {
      Slot sl = load_slot(tb, cfg.slot);
      if (cfg.lexnode != kNoLex && cfg.lexnode >= sl.nodes) b = 1;
    }
    bad = b;
    overflow = 0;
    nG = 0;
    winner = -1;
  }
  if (tid < 8) {
    A[tid] = 0;
    Aw[tid] = 0;
    uint32_t iw = 0, all = 0;
    for (int j = 0; j < 32; ++j) {
      const int t = tid * 32 + j;
      if (t < tb.T) {
        all |= 1u << j;
        if (tb.term_info[t] & 1u) iw |= 1u << j;
      }
    }
    I[tid] = iw;
    ALL[tid] = all;
  }
  if (grp == 0)
    for (int w = tid; w < tb.W; w += kBlock) mrow[w] = 0u;
  __syncthreads();
  const uint32_t depth = cfg.stk_depth;
  const uint32_t lo = depth > (uint32_t)kStackWin ? depth - kStackWin : 0;
  if (!bad) {
    for (uint32_t i = tid; i < depth; i += kBlock) {
      const uint16_t s = pool[cfg.stk_off + i];
      if (s >= tb.NS) bad = 1;
      if (i >= lo) win[i - lo] = s;
    }
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) {
      hdr->pstat[grp] = grp == 0 ? GRID_ROW_BAD_CONFIG : 0;
      if (grp == 0) {
        hdr->valid = 0;
        hdr->eos_ok = 0;
        hdr->slow_count = 0;
        hdr->wstat = 0;
        if (eos_out) eos_out[row] = 0;
      }
    }
    return;
  }
  const BaseStack bs{pool + cfg.stk_off, win, depth, lo};
  uint16_t* my = scratch[tid];

  // A(sigma): one set simulation over every terminal
  if (tid == 0) {
    uint32_t X[MW], acc[MW];
#pragma unroll
    for (int w = 0; w < MW; ++w) {
      X[w] = ALL[w];
      acc[w] = 0;
    }
    if (sim_set<MW>(pt, bs, depth, 0, my, my, kPostCap + kTmpCap, X, acc) < 0) overflow = 1;
#pragma unroll
    for (int w = 0; w < MW; ++w) A[w] = acc[w] & ALL[w];
    // the pending lexeme's winner if a byte ends it: the highest-priority
    // candidate that is allowed (or ignored) and passes the schema lexicon
    if (!(cfg.flags & 1u)) {
      const Slot sl = load_slot(tb, cfg.slot);
      const uint32_t lf = lex_flags_of(tb, sl, cfg.lexnode);
      for (uint32_t j = tb.acc_off[cfg.q]; j < tb.acc_off[cfg.q + 1]; ++j) {
        const int t = tb.acc_list[j];
        const uint32_t ti = tb.term_info[t];
        uint32_t c;
        const bool allowed = (ti & 1u) || ((A[t >> 5] >> (t & 31)) & 1u);
        const bool lexok = !restricted_cat(sl, ti, c) || ((lf >> (8 + c)) & 1u);
        if (allowed && lexok) {
          winner = t;
          break;
        }
      }
    }
    // terminals t of A with t mod kProGroups == grp; workgroup 0 also needs
    // the winner's stack and allowed set
    int n = 0;
    for (int t = grp; t < tb.T; t += kProGroups)
      if ((A[t >> 5] >> (t & 31)) & 1u) glist[n++] = (uint8_t)t;
    const int wt = winner;
    if (grp == 0 && wt >= 0 && wt % kProGroups != 0 && ((A[wt >> 5] >> (wt & 31)) & 1u)) glist[n++] = (uint8_t)wt;
    nG = n;
  }
  for (int i = tid; i < 256 * 8; i += kBlock) A2s[i] = 0;
  __syncthreads();
  // the stack after each allowed terminal's shift, then its allowed set
  for (int i = tid; i < nG; i += kBlock) {
    const int t = glist[i];
    uint32_t k = depth;
    int m = 0;
    const int r = sim1_shift(pt, bs, k, m, my, kPostCap, t);
    Post p;
    p.k = (uint16_t)k;
    p.m = (uint8_t)m;
    p.ok = r == 1;
    for (int j = 0; j < kPostCap; ++j) p.ov[j] = j < m ? my[j] : 0;
    if (r != 1 || k > 0xFFFF) overflow = 1;
    posts[t] = p;
    if (t % kProGroups == grp) post[t] = p;
    if (r == 1) {
      uint32_t X[MW], acc[MW];
#pragma unroll
      for (int w = 0; w < MW; ++w) {
        X[w] = ALL[w];
        acc[w] = 0;
      }
      if (sim_set<MW>(pt, bs, k, m, my, my + m, kPostCap + kTmpCap - m, X, acc) < 0) overflow = 1;
#pragma unroll
      for (int w = 0; w < MW; ++w) A2s[t * 8 + w] = acc[w] & ALL[w];
    }
  }
  __syncthreads();
  {  // allowed sets and trailing codes after this workgroup's first shifts
    const Slot sl0 = load_slot(tb, cfg.slot);
    uint16_t* vend1 = (uint16_t*)(rw + L.vend1);
    for (int i = tid; i < nG * 8; i += kBlock) {
      const int t = glist[i >> 3];
      if (t % kProGroups == grp) a2[t * 8 + (i & 7)] = A2s[t * 8 + (i & 7)];
    }
    const int n = nG * tb.S;
    for (int idx = tid; idx < n; idx += kBlock) {
      const int t = glist[idx / tb.S], q = idx % tb.S;
      if (t % kProGroups == grp) vend1[(size_t)t * L.s_pad + q] = state_code(tb, sl0, q, &A2s[t * 8], I);
    }
  }
  if (grp != 0) {
    __syncthreads();
    if (tid == 0) hdr->pstat[grp] = overflow ? GRID_ROW_OVERFLOW : 0;
    return;
  }

  // ---- workgroup 0: pending lexeme, EOS gate, state codes, first-byte table
  const Slot sl = load_slot(tb, cfg.slot);
  const bool rem_empty = (cfg.flags & 1u) != 0;
  const int w = winner;
  const bool w_shifts = w >= 0 && !(tb.term_info[w] & 1u);
  if (w_shifts && tid < 8) Aw[tid] = A2s[w * 8 + tid];
  __syncthreads();
  uint16_t* vend = (uint16_t*)(rw + L.vend);
  for (int q = tid; q < tb.S; q += kBlock) vend[q] = state_code(tb, sl, q, A, I);
  // first-byte table
  uint2* fb = (uint2*)(rw + L.fb);
  {
    const int b = tid;  // kBlock == 256: one byte value per thread
    const uint32_t c = tb.bclass[b];
    uint32_t kind = kFbDead, q1 = 0, t1 = 0, lex1 = kNoLex;
    const int nq = tb.dfa[(size_t)cfg.q * tb.C + c];
    if (nq != kDead) {
      lex1 = lex_child(tb, sl, cfg.lexnode, b);
      if (code_ok(state_code(tb, sl, nq, A, I), lex_flags_of(tb, sl, lex1))) {
        kind = kFbMode0;
        q1 = nq;
      }
    } else if (!rem_empty && w >= 0) {
      const int sq = tb.dfa[(size_t)kStart * tb.C + c];
      if (sq != kDead) {
        lex1 = lex_child(tb, sl, 0u, b);
        const uint32_t lf1 = lex_flags_of(tb, sl, lex1);
        if (!w_shifts) {
          if (code_ok(state_code(tb, sl, sq, A, I), lf1)) kind = kFbMode0;
        } else if (code_ok(state_code(tb, sl, sq, Aw, I), lf1)) {
          kind = kFbMode1;
          t1 = (uint32_t)w;
        }
        q1 = sq;
      }
    }
    if (kind == kFbDead) lex1 = kNoLex;
    fb[b] = make_uint2(q1 | kind << 16 | t1 << 24, lex1);
  }
  // end-of-sequence gate (mid-lexeme aware)
  if (tid == 0) {
    int ok = 0;
    if (rem_empty || (w >= 0 && !w_shifts)) {
      ok = sim1_test(pt, bs, depth, 0, my, my, kPostCap + kTmpCap, tb.T) == 2;
    } else if (w >= 0) {
      const Post& p = posts[w];
      ok = sim1_test(pt, bs, p.k, p.m, p.ov, my, kPostCap + kTmpCap, tb.T) == 2;
    }
    hdr->eos_ok = (uint32_t)ok;
    if (eos_out) eos_out[row] = (uint8_t)ok;
    if (ok && tb.eos_id >= 0) mrow[tb.eos_id >> 5] |= 1u << (tb.eos_id & 31);
  }
  __syncthreads();
  if (tid < 8) hdr->A[tid] = A[tid];
  if (tid == 0) {
    hdr->winner = w;
    hdr->slow_count = 0;
    hdr->wstat = 0;
    hdr->pstat[0] = overflow ? GRID_ROW_OVERFLOW : GRID_ROW_OK;
    hdr->valid = kRowValid;
  }
}

// ------------------------------------------------------- lane machinery
// Lane state after at least one byte: the stack is sigma (mode 0), the stack
// after the first shift t1 (mode 1), or base[0,k) ++ ov[0,m) (mode 2).
struct LaneState {
  int mode;
  int t1;
  uint32_t k;
  int m;
};

struct RowCtx {
  const Tables* tb;
  ParseTabs pt;
  BaseStack bs;
  Slot sl;
  const uint32_t* A;        // allowed set of sigma (8 words)
  const uint32_t* I;        // ignored terminals (8 words)
  const uint32_t* a2;       // row's A2 table (global)
  const Post* post;         // row's post table (global)
  const uint32_t* tinfo;    // terminal info (LDS or global)
  const uint32_t* acc_off;  // accept-list offsets (LDS or global)
  const uint8_t* acc_list;  // accept lists (LDS or global)
  const uint16_t* vend0;    // trailing codes under A(sigma)
  const uint16_t* vendw;    // trailing codes after the row winner's shift
  const uint16_t* vend1;    // trailing codes after each first shift, [T][s_pad] (global)
  size_t s_pad;
  int winner;
};

// Trailing-code row for a lane in mode 0 or 1.
__device__ inline const uint16_t* code_row(const RowCtx& rc, const LaneState& st) {
  if (st.mode == 0) return rc.vend0;
  if (st.t1 == rc.winner) return rc.vendw;
  return rc.vend1 + (size_t)st.t1 * rc.s_pad;
}

// Emits the pending lexeme in DFA state q (lexicon flags lf).  ov is the
// lane's stack area of cap entries: the overlay occupies [0, m), virtual
// pushes use [m, cap).  1 ok, 0 reject, -1 capacity.
template <int MW>
__device__ int emit_general(const RowCtx& rc, LaneState& st, uint16_t* ov, int cap, int q, uint32_t lf) {
  const uint32_t a0 = rc.acc_off[q], a1 = rc.acc_off[q + 1];
  if (a0 == a1) return 0;
  uint32_t acc[MW];
#pragma unroll
  for (int w = 0; w < MW; ++w) acc[w] = 0;
  if (st.mode == 2) {  // one set simulation over the non-ignored candidates
    uint32_t X[MW];
#pragma unroll
    for (int w = 0; w < MW; ++w) X[w] = 0;
    for (uint32_t j = a0; j < a1; ++j) {
      const int t = rc.acc_list[j];
      const uint32_t ti = rc.tinfo[t];
      uint32_t c;
      if ((ti & 1u) || (restricted_cat(rc.sl, ti, c) && !((lf >> (8 + c)) & 1u))) continue;
#pragma unroll
      for (int w = 0; w < MW; ++w)
        if (w == (t >> 5)) X[w] |= 1u << (t & 31);
    }
    if (sim_set<MW>(rc.pt, rc.bs, st.k, st.m, ov, ov + st.m, cap - st.m, X, acc) < 0) return -1;
  }
  int winner = -1;
  for (uint32_t j = a0; j < a1; ++j) {
    const int t = rc.acc_list[j];
    const uint32_t ti = rc.tinfo[t];
    uint32_t c;
    if (restricted_cat(rc.sl, ti, c) && !((lf >> (8 + c)) & 1u)) continue;
    bool ok;
    if (ti & 1u) ok = true;
    else if (st.mode == 0) ok = (rc.A[t >> 5] >> (t & 31)) & 1u;
    else if (st.mode == 1) ok = (rc.a2[st.t1 * 8 + (t >> 5)] >> (t & 31)) & 1u;
    else {
      ok = false;
#pragma unroll
      for (int w = 0; w < MW; ++w)
        if (w == (t >> 5)) ok = (acc[w] >> (t & 31)) & 1u;
    }
    if (ok) {
      winner = t;
      break;
    }
  }
  if (winner < 0) return 0;
  if (rc.tinfo[winner] & 1u) return 1;  // ignored: the stack is unchanged
  if (st.mode == 0) {
    st.mode = 1;
    st.t1 = winner;
    return 1;
  }
  if (st.mode == 1) {
    const Post& p = rc.post[st.t1];
    if (p.k == 0 || p.k > rc.bs.depth || p.m > kPostCap || p.m > cap) return -1;
    st.k = p.k;
    st.m = p.m;
    for (int j = 0; j < st.m; ++j) ov[j] = p.ov[j];
    st.mode = 2;
  }
  const int r = sim1_shift(rc.pt, rc.bs, st.k, st.m, ov, cap, winner);
  return r < 0 ? -1 : (r == 1);
}

// Trailing test of Definition 2 in any lane state.  -1: capacity.
template <int MW>
__device__ int trailing_any(const RowCtx& rc, const LaneState& st, uint16_t* ov, int cap, int q, uint32_t lex) {
  const Tables& tb = *rc.tb;
  if (st.mode <= 1) {
    const uint32_t code = code_row(rc, st)[q];
    if (code & 0x8000u) return 1;
    if (!(code & 0xFFu)) return 0;
    return (lex_flags_of(tb, rc.sl, lex) & code & 0xFFu) != 0;
  }
  const uint32_t lf = lex_flags_of(tb, rc.sl, lex);
  uint32_t X[MW], any = 0;
#pragma unroll
  for (int w = 0; w < MW; ++w) {
    uint32_t bits = tb.live[(size_t)q * 8 + w];
    uint32_t keep = 0;
    while (bits) {
      const int b = __ffs(bits) - 1;
      bits &= bits - 1;
      const int t = w * 32 + b;
      const uint32_t ti = rc.tinfo[t];
      uint32_t c;
      if (restricted_cat(rc.sl, ti, c) && !((lf >> c) & 1u)) continue;
      if (ti & 1u) return 1;
      keep |= 1u << b;
    }
    X[w] = keep;
    any |= keep;
  }
  if (!any) return 0;
  uint32_t acc[MW];
#pragma unroll
  for (int w = 0; w < MW; ++w) acc[w] = 0;
  if (sim_set<MW>(rc.pt, rc.bs, st.k, st.m, ov, ov + st.m, cap - st.m, X, acc) < 0) return -1;
  uint32_t hit = 0;
#pragma unroll
  for (int w = 0; w < MW; ++w) hit |= acc[w] & X[w];
  return hit != 0;
}

__device__ inline void set_alias_bits(const Tables& tb, uint32_t* mrow, int u) {
  for (uint32_t j = tb.alias_off[u]; j < tb.alias_off[u + 1]; ++j) {
    const int id = tb.alias_ids[j];
    atomicOr(&mrow[id >> 5], 1u << (id & 31));
  }
}

struct DfaView {  // lexer DFA by byte class (LDS copy or global)
  const uint16_t* next_;
  const uint8_t* cls_;
  int C;
  __device__ uint32_t cls(uint32_t b) const { return cls_[b]; }
  __device__ int next(int q, uint32_t c) const { return next_[q * C + c]; }
};

// Walks the bytes [i, n) of one spelling from lane state (st, q, lex).
// byte_at(i) yields byte i.  1 allowed, 0 rejected, -1 capacity.
template <int MW, class ByteAt>
__device__ inline int walk_bytes(const RowCtx& rc, LaneState& st, int q, uint32_t lex, uint32_t i, uint32_t n,
                                 ByteAt byte_at, const DfaView& step, uint16_t* ov, int cap) {
  const Tables& tb = *rc.tb;
  for (; i < n; ++i) {
    const uint32_t b = byte_at(i);
    const uint32_t c = step.cls(b);
    const int nq = step.next(q, c);
    if (nq != kDead) {
      q = nq;
      if (lex != kNoLex) lex = lex_child(tb, rc.sl, lex, b);
    } else {
      const int r = emit_general<MW>(rc, st, ov, cap, q, lex_flags_of(tb, rc.sl, lex));
      if (r <= 0) return r;
      q = step.next(kStart, c);
      if (q == kDead) return 0;
      lex = lex_child(tb, rc.sl, 0u, b);
    }
    const int r = trailing_any<MW>(rc, st, ov, cap, q, lex);
    if (r <= 0) return r;
  }
  return 1;
}

// -------------------------------------------------------------------- walk
struct WalkLds {  // byte offsets into dynamic LDS
  uint32_t dfa, bcls, tinfo, I, acc_off, acc_list, parse, fb, vend0, vendw, lanes, total, vstride;
  ParseLds pl;
};

__host__ __device__ inline WalkLds walk_lds(const Tables& tb) {
  WalkLds w;
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
  w.pl = parse_lds(tb, o);
  o += w.pl.total;
  w.fb = o;
  o += 256 * 8;
  w.vstride = pad16((uint32_t)((tb.S + 7) & ~7) * 2);
  w.vend0 = o;
  o += w.vstride;
  w.vendw = o;
  o += w.vstride;
  w.lanes = o;
  o += kWalkThreads * kFastLane * 2;
  w.total = o;
  return w;
}

// Persistent: each workgroup stages the grammar tables once, then takes work
// items (row x spelling tile) from a counter in the workspace head.
template <int MW>
__global__ __launch_bounds__(kWalkThreads) void walk_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                            const uint16_t* __restrict__ pool,
                                                            uint32_t* __restrict__ mask,
                                                            uint8_t* __restrict__ ws, size_t rbytes, int B,
                                                            int n_tiles, int n_items) {
  extern __shared__ __align__(16) uint8_t lds[];
  __shared__ int item_s;
  __shared__ uint32_t A_s[8];
  __shared__ int winner_s;
  const int tid = threadIdx.x;
  const WalkLds WL = walk_lds(tb);
  const RowLayout RL = row_layout(tb.T, tb.S);
  uint8_t* bcls = lds + WL.bcls;
  uint32_t* tinfo_s = (uint32_t*)(lds + WL.tinfo);
  uint32_t* I_s = (uint32_t*)(lds + WL.I);
  uint2* fb_s = (uint2*)(lds + WL.fb);
  uint16_t* lane = (uint16_t*)(lds + WL.lanes) + tid * kFastLane;
  uint32_t* counter = (uint32_t*)ws;
  uint8_t* rows = ws + kWsHead;

  // grammar tables, once per workgroup
  stage16(lds + WL.dfa, (const uint8_t*)tb.dfa, (uint32_t)(tb.S * tb.C * 2), tid, kWalkThreads);
  stage16(bcls, tb.bclass, 256, tid, kWalkThreads);
  stage16(lds + WL.acc_off, (const uint8_t*)tb.acc_off, (uint32_t)(tb.S + 1) * 4, tid, kWalkThreads);
  stage16(lds + WL.acc_list, tb.acc_list, (uint32_t)tb.n_acc, tid, kWalkThreads);
  const ParseTabs pt = stage_parse(tb, lds, WL.pl, tid, kWalkThreads);
  for (int t = tid; t < 256; t += kWalkThreads) tinfo_s[t] = t < tb.T ? tb.term_info[t] : 0u;
  __syncthreads();
  if (tid < 8) {
    uint32_t iw = 0;
    for (int j = 0; j < 32; ++j)
      if (tinfo_s[tid * 32 + j] & 1u) iw |= 1u << j;
    I_s[tid] = iw;
  }

  const DfaView step{(const uint16_t*)(lds + WL.dfa), bcls, tb.C};
  const uint4* recs = tb.spell_rec;
  for (;;) {
    __syncthreads();  // the previous item is done with the row tables
    if (tid == 0) item_s = (int)atomicAdd(counter, 1u);
    __syncthreads();
    const int item = item_s;
    if (item >= n_items) break;
    const int row = item / n_tiles;
    const int tile = item % n_tiles;
    uint8_t* rw = rows + (size_t)row * rbytes;
    RowHeader* hdr = (RowHeader*)rw;
    if (hdr->valid != kRowValid) continue;  // uniform across the workgroup
    const int w = hdr->winner;
    const bool w_shifts = w >= 0 && !(tinfo_s[w] & 1u);
    stage16((uint8_t*)fb_s, rw + RL.fb, 256 * 8, tid, kWalkThreads);
    stage16(lds + WL.vend0, rw + RL.vend, WL.vstride, tid, kWalkThreads);
    if (w_shifts)
      stage16(lds + WL.vendw, rw + RL.vend1 + (size_t)w * RL.s_pad * 2, WL.vstride, tid, kWalkThreads);
    if (tid < 8) A_s[tid] = hdr->A[tid];
    if (tid == 0) winner_s = w_shifts ? w : -1;
    __syncthreads();

    // this thread's spellings in the tile
    static_assert(kWalkSpt == 2, "two spelling records per thread");
    const int ubase = tile * kWalkTile + tid;
    const uint4 rec0 = ubase < tb.U ? recs[ubase] : make_uint4(0, 0, 0, 0);
    const uint4 rec1 = ubase + kWalkThreads < tb.U ? recs[ubase + kWalkThreads] : make_uint4(0, 0, 0, 0);
    const grid_config cfg = cfgs[row];
    RowCtx rc;
    rc.tb = &tb;
    rc.pt = pt;
    rc.bs = BaseStack{pool + cfg.stk_off, nullptr, cfg.stk_depth, cfg.stk_depth};
    rc.sl = load_slot(tb, cfg.slot);
    rc.A = A_s;
    rc.I = I_s;
    rc.a2 = (const uint32_t*)(rw + RL.a2);
    rc.post = (const Post*)(rw + RL.post);
    rc.tinfo = tinfo_s;
    rc.acc_off = (const uint32_t*)(lds + WL.acc_off);
    rc.acc_list = lds + WL.acc_list;
    rc.vend0 = (const uint16_t*)(lds + WL.vend0);
    rc.vendw = (const uint16_t*)(lds + WL.vendw);
    rc.vend1 = (const uint16_t*)(rw + RL.vend1);
    rc.s_pad = RL.s_pad;
    rc.winner = winner_s;
    uint32_t* mrow = mask + (size_t)row * tb.W;
    int handoff = 0;

#pragma unroll 1
    for (int k = 0; k < kWalkSpt; ++k) {
      const uint4 rk = k == 0 ? rec0 : rec1;
      const uint32_t n = rk.w;
      if (n == 0) continue;
      const uint64_t h = (uint64_t)rk.x | (uint64_t)rk.y << 32;
      const uint2 e = fb_s[h & 0xFF];
      const uint32_t kind = (e.x >> 16) & 3u;
      if (kind == kFbDead) continue;
      const int u = ubase + k * kWalkThreads;
      LaneState st{(int)kind - 1, (int)(e.x >> 24), 0, 0};
      uint32_t off = 0;
      auto byte_at = [&](uint32_t i) -> uint32_t {
        if (i < 8) return (uint32_t)(h >> (8 * i)) & 0xFFu;
        if (i == 8) off = tb.spell_off[u];
        return tb.spell_bytes[off + i];
      };
      const int ok = walk_bytes<MW>(rc, st, (int)(e.x & 0xFFFF), e.y, 1u, n, byte_at, step, lane, kFastLane);
      if (ok > 0) {
        const uint32_t id = rk.z;
        if (!(id >> 31)) atomicOr(&mrow[id >> 5], 1u << (id & 31));
        else set_alias_bits(tb, mrow, u);
      } else if (ok < 0) {  // the lane's stack area is too small: hand over
        const uint32_t slot = atomicAdd(&hdr->slow_count, 1u);
        if (slot < (uint32_t)kSlowCap) ((uint32_t*)(rw + RL.slow))[slot] = (uint32_t)u;
        else handoff = 1;
      }
    }
    if (handoff) atomicOr(&hdr->wstat, GRID_ROW_OVERFLOW);
  }
}

// ---------------------------------------------------------------- finalize
// Re-walks handed-over spellings from the row's configuration with a large
// stack area in the workspace, then combines the status bits.
template <int MW>
__global__ __launch_bounds__(kSlowThreads) void finalize_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                                const uint16_t* __restrict__ pool,
                                                                uint32_t* __restrict__ mask,
                                                                uint8_t* __restrict__ ws, size_t rbytes,
                                                                int32_t* __restrict__ status) {
  extern __shared__ __align__(16) uint8_t flds[];
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  uint8_t* rw = ws + kWsHead + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  const RowLayout RL = row_layout(tb.T, tb.S);
  uint32_t* mrow = mask + (size_t)row * tb.W;
  __shared__ uint32_t any;
  __shared__ int slow_err;
  __shared__ uint32_t I_s[8];
  if (tid == 0) {
    any = 0;
    slow_err = 0;
  }
  if (tid < 8) {
    uint32_t iw = 0;
    for (int j = 0; j < 32; ++j) {
      const int t = tid * 32 + j;
      if (t < tb.T && (tb.term_info[t] & 1u)) iw |= 1u << j;
    }
    I_s[tid] = iw;
  }
  const bool valid = hdr->valid == kRowValid;
  const uint32_t count = valid ? min(hdr->slow_count, (uint32_t)kSlowCap) : 0u;
  ParseTabs pt = global_parse(tb);
  if (count > 0) pt = stage_parse(tb, flds, parse_lds(tb, 0), tid, kSlowThreads);
  __syncthreads();
  if (count > 0) {
    const grid_config cfg = cfgs[row];
    RowCtx rc;
    rc.tb = &tb;
    rc.pt = pt;
    rc.bs = BaseStack{pool + cfg.stk_off, nullptr, cfg.stk_depth, cfg.stk_depth};
    rc.sl = load_slot(tb, cfg.slot);
    rc.A = hdr->A;
    rc.I = I_s;
    rc.a2 = (const uint32_t*)(rw + RL.a2);
    rc.post = (const Post*)(rw + RL.post);
    rc.tinfo = tb.term_info;
    rc.acc_off = tb.acc_off;
    rc.acc_list = tb.acc_list;
    rc.vend0 = (const uint16_t*)(rw + RL.vend);
    rc.vend1 = (const uint16_t*)(rw + RL.vend1);
    rc.s_pad = RL.s_pad;
    rc.winner = -1;  // every mode-1 lane reads its own trailing-code row
    rc.vendw = rc.vend1;
    uint16_t* ov = (uint16_t*)(rw + RL.slow_ov) + tid * kSlowLane;
    const DfaView step{tb.dfa, tb.bclass, tb.C};
    for (uint32_t k = tid; k < count; k += kSlowThreads) {
      const int u = (int)((const uint32_t*)(rw + RL.slow))[k];
      LaneState st{0, -1, 0, 0};
      const uint32_t base = tb.spell_off[u];
      auto byte_at = [&](uint32_t i) -> uint32_t { return tb.spell_bytes[base + i]; };
      const int ok = walk_bytes<MW>(rc, st, cfg.q, cfg.lexnode, 0u, tb.spell_off[u + 1] - base, byte_at, step, ov,
                                    kSlowLane);
      if (ok > 0) set_alias_bits(tb, mrow, u);
      if (ok < 0) slow_err = 1;
    }
  }
  __syncthreads();
  __threadfence();
  uint32_t acc = 0;
  for (int w = tid; w < tb.W; w += kSlowThreads) acc |= __atomic_load_n(&mrow[w], __ATOMIC_RELAXED);
  if (acc) atomicOr(&any, 1u);
  __syncthreads();
  if (tid == 0) {
    int32_t st = 0;
    if (valid) {
      for (int g = 0; g < kProGroups; ++g) st |= hdr->pstat[g];
      st |= hdr->wstat;
      if (slow_err || hdr->slow_count > (uint32_t)kSlowCap) st |= GRID_ROW_OVERFLOW;
      if (!any && !hdr->eos_ok) st |= GRID_ROW_EMPTY;
    } else {
      st = hdr->pstat[0] | GRID_ROW_BAD_CONFIG;
    }
    if (status) status[row] = st;
  }
}

// ------------------------------------------------------------------- apply
// Each thread covers 8 consecutive logits of one row; the mask byte for them
// comes from one word.  Fully masked groups take one or two 16-byte stores.
template <typename T>
__global__ __launch_bounds__(kBlock) void apply_kernel(const uint32_t* __restrict__ mask, T* logits, int B,
                                                       int V, int W, int64_t stride, uint32_t neg_inf_bits,
                                                       bool vec_ok) {
  const int groups = (V + 7) >> 3;
  const int64_t total = (int64_t)B * groups;
  for (int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x; g < total;
       g += (int64_t)gridDim.x * kBlock) {
    const int row = (int)(g / groups);
    const int col = (int)(g - (int64_t)row * groups) * 8;
    const uint32_t bits = (mask[(size_t)row * W + (col >> 5)] >> (col & 31)) & 0xFFu;
    if (bits == 0xFFu) continue;
    T* p = logits + row * stride + col;
    if (bits == 0 && col + 8 <= V && vec_ok) {
      if (sizeof(T) == 2) {
        const uint32_t w2 = neg_inf_bits | (neg_inf_bits << 16);
        *reinterpret_cast<uint4*>(p) = make_uint4(w2, w2, w2, w2);
      } else {
        const uint4 v = make_uint4(neg_inf_bits, neg_inf_bits, neg_inf_bits, neg_inf_bits);
        reinterpret_cast<uint4*>(p)[0] = v;
        reinterpret_cast<uint4*>(p)[1] = v;
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

bool bound(const grid_compiled* g, int which) { return g->dev[which] != nullptr || g->dev_bytes[which] == 0; }

// Resident walk workgroups per device (compute units x occupancy), cached.
template <int MW>
int walk_grid_size(size_t lds) {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] > 0) return cached[dev];
  int cus = 0, per_cu = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0) cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, walk_kernel<MW>, kWalkThreads, lds) != hipSuccess ||
      per_cu <= 0)
    per_cu = 1;
  cached[dev] = cus * per_cu;
  return cached[dev];
}

template <int MW>
void launch_mask(const Tables& tb, int B, const grid_config* cfg_dev, const uint16_t* pool, uint32_t* mask,
                 uint8_t* eos, int32_t* status, uint8_t* ws, size_t rb, uint32_t phases, hipStream_t s) {
  const uint32_t parse_bytes = parse_lds(tb, 0).total;
  if (phases & GRID_PHASE_PROLOGUE)
    hipLaunchKernelGGL(prologue_kernel<MW>, dim3(B, kProGroups), dim3(kBlock), parse_bytes, s, tb, cfg_dev, pool,
                       mask, eos, ws, rb);
  if ((phases & GRID_PHASE_WALK) && tb.U > 0) {
    const WalkLds WL = walk_lds(tb);
    const int n_tiles = (tb.U + kWalkTile - 1) / kWalkTile;
    const int n_items = n_tiles * B;
    const int blocks = std::min(n_items, walk_grid_size<MW>(WL.total));
    hipLaunchKernelGGL(walk_kernel<MW>, dim3(blocks), dim3(kWalkThreads), WL.total, s, tb, cfg_dev, pool, mask, ws,
                       rb, B, n_tiles, n_items);
  }
  if (phases & GRID_PHASE_FINALIZE)
    hipLaunchKernelGGL(finalize_kernel<MW>, dim3(B), dim3(kSlowThreads), parse_bytes, s, tb, cfg_dev, pool, mask,
                       ws, rb, status);
}

}  // namespace

int grid::overlay_capacity() { return kFastLane; }

extern "C" size_t grid_mask_workspace_bytes(const grid_compiled* g, int32_t B) {
  if (!g || B <= 0) return 0;
  return kWsHead + row_layout(g->parser.T, g->dfa.S).total * (size_t)B;
}

extern "C" int grid_mask_phases(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                                const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                                int32_t* status_dev, void* workspace_dev, size_t workspace_bytes,
                                uint32_t phases, void* stream) {
  clear_error();
  if (phases & ~GRID_PHASE_ALL) return fail(GRID_E_ARG, "grid_mask: unknown phase bits");
  if (!g || B <= 0 || B > 65535 || !cfg_dev || !stack_pool_dev || !mask_dev || !workspace_dev)
    return fail(GRID_E_ARG, "grid_mask: null pointer or batch size out of range");
  const size_t rb = row_layout(g->parser.T, g->dfa.S).total;
  if (workspace_bytes < kWsHead + rb * (size_t)B) return fail(GRID_E_ARG, "grid_mask: workspace too small");
  if (((uintptr_t)workspace_dev & 255) != 0) return fail(GRID_E_ARG, "grid_mask: workspace not 256-byte aligned");
  static const int needed[] = {GRID_ART_DFA_CLASS,  GRID_ART_BYTE_CLASS, GRID_ART_DFA_ACCEPT_OFF,
                               GRID_ART_DFA_ACCEPT_LIST, GRID_ART_DFA_LIVE, GRID_ART_ACTION,
                               GRID_ART_PROD,       GRID_ART_TERM_INFO,  GRID_ART_SPELL_OFF,
                               GRID_ART_SPELL_BYTES, GRID_ART_SPELL_REC, GRID_ART_ALIAS_OFF,
                               GRID_ART_ALIAS_IDS,  GRID_ART_LEX_FLAGS,  GRID_ART_LEX_HASH,
                               GRID_ART_LEX_SLOTS,  GRID_ART_PARSE_STATE, GRID_ART_PARSE_REDX,
                               GRID_ART_GOTO_OFF,   GRID_ART_GOTO_ENT};
  for (int w : needed)
    if (!bound(g, w)) return fail(GRID_E_UNBOUND, "grid_mask: artifact " + std::to_string(w) + " is not bound");
  Tables tb;
  tb.dfa = (const uint16_t*)g->dev[GRID_ART_DFA_CLASS];
  tb.bclass = (const uint8_t*)g->dev[GRID_ART_BYTE_CLASS];
  tb.acc_off = (const uint32_t*)g->dev[GRID_ART_DFA_ACCEPT_OFF];
  tb.acc_list = (const uint8_t*)g->dev[GRID_ART_DFA_ACCEPT_LIST];
  tb.live = (const uint32_t*)g->dev[GRID_ART_DFA_LIVE];
  tb.action = (const uint16_t*)g->dev[GRID_ART_ACTION];
  tb.prod = (const uint32_t*)g->dev[GRID_ART_PROD];
  tb.term_info = (const uint32_t*)g->dev[GRID_ART_TERM_INFO];
  tb.pstate = (const uint32_t*)g->dev[GRID_ART_PARSE_STATE];
  tb.predx = (const uint32_t*)g->dev[GRID_ART_PARSE_REDX];
  tb.goff = (const uint32_t*)g->dev[GRID_ART_GOTO_OFF];
  tb.gent = (const uint32_t*)g->dev[GRID_ART_GOTO_ENT];
  tb.spell_off = (const uint32_t*)g->dev[GRID_ART_SPELL_OFF];
  tb.spell_bytes = (const uint8_t*)g->dev[GRID_ART_SPELL_BYTES];
  tb.spell_rec = (const uint4*)g->dev[GRID_ART_SPELL_REC];
  tb.alias_off = (const uint32_t*)g->dev[GRID_ART_ALIAS_OFF];
  tb.alias_ids = (const int32_t*)g->dev[GRID_ART_ALIAS_IDS];
  tb.lex_flags = (const uint16_t*)g->dev[GRID_ART_LEX_FLAGS];
  tb.lex_hash = (const uint32_t*)g->dev[GRID_ART_LEX_HASH];
  tb.lex_slots = (const uint32_t*)g->dev[GRID_ART_LEX_SLOTS];
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
  tb.n_gent = (int)g->parser.goto_ent.size();
  tb.n_acc = (int)g->dfa.accept_list.size();
  const WalkLds WL = walk_lds(tb);
  if (WL.total > 64 * 1024 || tb.n_acc > kAccCap || parse_lds(tb, 0).total > 32 * 1024 || tb.tw > 8)
    return fail(GRID_E_CAPACITY, "grid_mask: lexer DFA or LR tables too large for the LDS staging");
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace_dev;
  if (tb.tw <= 4)
    launch_mask<4>(tb, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, ws, rb, phases, s);
  else
    launch_mask<8>(tb, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, ws, rb, phases, s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_mask launch: ") + hipGetErrorString(e));
  return GRID_OK;
}

extern "C" int grid_mask(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                         const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                         int32_t* status_dev, void* workspace_dev, size_t workspace_bytes, void* stream) {
  return grid_mask_phases(g, B, cfg_dev, stack_pool_dev, mask_dev, eos_dev, status_dev, workspace_dev,
                          workspace_bytes, GRID_PHASE_ALL, stream);
}

extern "C" int grid_apply(const uint32_t* mask_dev, void* logits_dev, int32_t dtype, int32_t B, int32_t V,
                          int64_t row_stride, void* stream) {
  clear_error();
  if (!mask_dev || !logits_dev || B <= 0 || V <= 0 || row_stride < V)
    return fail(GRID_E_ARG, "grid_apply: null pointer or bad shape");
  if (dtype != GRID_DTYPE_F32 && dtype != GRID_DTYPE_BF16) return fail(GRID_E_ARG, "grid_apply: dtype");
  const int W = (V + 31) / 32;
  const int64_t groups = (int64_t)B * ((V + 7) / 8);
  const int blocks = (int)std::min<int64_t>((groups + kBlock - 1) / kBlock, 256 * 64);
  hipStream_t s = (hipStream_t)stream;
  const size_t esz = dtype == GRID_DTYPE_BF16 ? 2 : 4;
  const bool vec_ok = ((uintptr_t)logits_dev % 16 == 0) && ((row_stride * (int64_t)esz) % 16 == 0);
  if (dtype == GRID_DTYPE_BF16)
    hipLaunchKernelGGL(apply_kernel<uint16_t>, dim3(blocks), dim3(kBlock), 0, s, mask_dev,
                       (uint16_t*)logits_dev, B, V, W, row_stride, 0xFF80u, vec_ok);
  else
    hipLaunchKernelGGL(apply_kernel<uint32_t>, dim3(blocks), dim3(kBlock), 0, s, mask_dev,
                       (uint32_t*)logits_dev, B, V, W, row_stride, 0xFF800000u, vec_ok);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(GRID_E_HIP, std::string("grid_apply launch: ") + hipGetErrorString(e));
  return GRID_OK;
}
