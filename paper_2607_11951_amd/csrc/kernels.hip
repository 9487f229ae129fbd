// kernels.hip -- device side of the cold exact mask and the -inf apply (gfx950).
//
// grid_mask launches, on the caller's stream:
//  1. prologue (one workgroup per row): stages the top of the row's LR stack,
//     computes the allowed terminals A(sigma) by running each terminal's
//     reduce chain on a private overlay above the shared read-only stack
//     (section 3.2, allowed terminals under table compression), records for
//     every allowed terminal the stack after its shift and that stack's own
//     allowed set, the end-of-sequence gate (section 3.2, EOS gating,
//     mid-lexeme aware), and a per-DFA-state code for the trailing-lexeme test
//     of Definition 2 under A(sigma); clears the row's mask words;
//  2. walk (rows x spelling tiles): one lane per distinct spelling, bytes in
//     trie (byte) order so neighbouring lanes share prefixes and die together.
//     Bytes step the lexer DFA; a byte that kills it emits the pending lexeme
//     as the highest-priority candidate that is allowed (or ignored) and
//     passes the schema lexicon, then rescans the byte (section 4.1, trie
//     walk).  Tokens that never leave the pending lexeme are decided by the
//     per-state code (context-independent part, section 4.2); after a first
//     shift the recorded stack and allowed set are used, and later shifts
//     simulate reduce chains on the lane's own overlay (context-dependent
//     part, Proposition 4).  Rejection is monotone, so a lane stops at the
//     first failing byte.  Allowed spellings set the bits of every alias id;
//  3. finalize (one workgroup per row): row status, empty-mask detection
//     (Proposition 8: a viable configuration has a nonempty mask).
// grid_apply is a streaming in-place -inf fill of the masked logits.
#include <hip/hip_runtime.h>

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

constexpr int kBlock = 256;
constexpr int kOvCap = 48;          // per-lane overlay states above the shared base
constexpr int kTmpCap = 16;         // virtual pushes while testing one terminal
constexpr int kLaneWords = kOvCap + kTmpCap;
constexpr int kStackWin = 256;      // top of the row's stack kept in LDS
constexpr int kPostCap = 14;        // overlay states recorded per first shift
constexpr int kGuard = 4096;        // reduce-chain step bound
constexpr int kSpellPerBlock = 1024;
constexpr uint32_t kRowValid = 0x600D;

struct Tables {
  const uint16_t* dfa;        // [S*C]
  const uint8_t* bclass;      // [256]
  const uint32_t* acc_off;    // [S+1]
  const uint8_t* acc_list;
  const uint32_t* live;       // [S*8]
  const uint16_t* action;     // [NS*(T+1)]
  const uint16_t* go;         // [NS*N]
  const uint32_t* prod;
  const uint32_t* term_info;  // [T]
  const uint32_t* spell_off;  // [U+1]
  const uint8_t* spell_bytes;
  const uint32_t* alias_off;  // [U+1]
  const int32_t* alias_ids;
  const uint16_t* lex_flags;
  const uint32_t* lex_hash;
  const uint32_t* lex_slots;
  int S, C, T, N, NS, U, V, W, n_slots, eos_id;
};

// Workspace layout per row.
struct RowHeader {
  uint32_t A[8];
  uint32_t eos_ok;
  int32_t status;
  uint32_t valid;
  uint32_t pad[21];
};
static_assert(sizeof(RowHeader) == 128, "row header is 128 bytes");

struct Post {             // stack after shifting one allowed terminal
  uint16_t k;             // shared base entries kept
  uint8_t m;              // overlay entries
  uint8_t ok;
  uint16_t ov[kPostCap];
};
static_assert(sizeof(Post) == 32, "post entry is 32 bytes");

__host__ __device__ inline size_t row_bytes(int T, int S) {
  size_t b = sizeof(RowHeader) + (size_t)T * sizeof(Post) + (size_t)T * 32 + (size_t)S * 2;
  return (b + 255) & ~(size_t)255;
}
__device__ inline Post* row_post(uint8_t* r) { return (Post*)(r + sizeof(RowHeader)); }
__device__ inline uint32_t* row_a2(uint8_t* r, int T) {
  return (uint32_t*)(r + sizeof(RowHeader) + (size_t)T * sizeof(Post));
}
__device__ inline uint16_t* row_vend(uint8_t* r, int T) {
  return (uint16_t*)(r + sizeof(RowHeader) + (size_t)T * sizeof(Post) + (size_t)T * 32);
}

struct BaseStack {  // the shared read-only stack of one row
  const uint16_t* pool;  // states [0, depth)
  const uint16_t* win;   // LDS copy of states [lo, depth)
  uint32_t depth, lo;
  __device__ uint16_t at(uint32_t i) const { return i >= lo ? win[i - lo] : pool[i]; }
};

// Reduce chain of terminal x on base[0,k) ++ ov[0,m) without changing it.
// 1 shift, 2 accept, 0 error, -1 capacity.
__device__ int sim_test(const Tables& tb, const BaseStack& bs, uint32_t k, int m, const uint16_t* ov,
                        uint16_t* tmp, int x) {
  int t = 0;
  const int T1 = tb.T + 1;
  for (int guard = 0; guard < kGuard; ++guard) {
    uint16_t top = t > 0 ? tmp[t - 1] : (m > 0 ? ov[m - 1] : bs.at(k - 1));
    uint16_t a = tb.action[(size_t)top * T1 + x];
    if (a == 0) return 0;
    uint16_t kind = a & 0xC000;
    if (kind == kActShift) return 1;
    if (kind == kActAccept) return 2;
    uint32_t pr = tb.prod[a & 0x3FFF];
    uint32_t len = pr >> 16;
    uint32_t d = min((uint32_t)t, len);
    t -= (int)d;
    len -= d;
    d = min((uint32_t)m, len);
    m -= (int)d;
    len -= d;
    if (len >= k) return 0;
    k -= len;
    uint16_t under = t > 0 ? tmp[t - 1] : (m > 0 ? ov[m - 1] : bs.at(k - 1));
    uint16_t g = tb.go[(size_t)under * tb.N + (pr & 0xFFFF)];
    if (g == kNoGoto) return 0;
    if (t >= kTmpCap) return -1;
    tmp[t++] = g;
  }
  return -1;
}

// Reduce chain of terminal x applied to (k, m, ov), then the shift.
__device__ int sim_shift(const Tables& tb, const BaseStack& bs, uint32_t& k, int& m, uint16_t* ov,
                         int cap, int x) {
  const int T1 = tb.T + 1;
  for (int guard = 0; guard < kGuard; ++guard) {
    uint16_t top = m > 0 ? ov[m - 1] : bs.at(k - 1);
    uint16_t a = tb.action[(size_t)top * T1 + x];
    if (a == 0) return 0;
    uint16_t kind = a & 0xC000;
    if (kind == kActShift) {
      if (m >= cap) return -1;
      ov[m++] = (uint16_t)(a & 0x3FFF);
      return 1;
    }
    if (kind == kActAccept) return 2;
    uint32_t pr = tb.prod[a & 0x3FFF];
    uint32_t len = pr >> 16;
    uint32_t d = min((uint32_t)m, len);
    m -= (int)d;
    len -= d;
    if (len >= k) return 0;
    k -= len;
    uint16_t under = m > 0 ? ov[m - 1] : bs.at(k - 1);
    uint16_t g = tb.go[(size_t)under * tb.N + (pr & 0xFFFF)];
    if (g == kNoGoto) return 0;
    if (m >= cap) return -1;
    ov[m++] = g;
  }
  return -1;
}

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

// ---------------------------------------------------------------- prologue
__global__ __launch_bounds__(kBlock) void prologue_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                          const uint16_t* __restrict__ pool,
                                                          uint32_t* __restrict__ mask,
                                                          uint8_t* __restrict__ eos_out,
                                                          uint8_t* __restrict__ ws, size_t rbytes) {
  const int row = blockIdx.x;
  const int tid = threadIdx.x;
  __shared__ uint16_t win[kStackWin];
  __shared__ uint32_t A[8], I[8];
  __shared__ uint32_t A2s[256 * 8];
  __shared__ uint16_t scratch[kBlock][kPostCap + kTmpCap];
  __shared__ uint8_t alist[256];
  __shared__ int nA, bad, overflow;
  uint8_t* rw = ws + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  const grid_config cfg = cfgs[row];
  uint32_t* mrow = mask + (size_t)row * tb.W;

  if (tid == 0) {
    int b = 0;
    if (cfg.q >= tb.S || cfg.slot >= tb.n_slots || cfg.stk_depth < 1) b = 1;
    if (!b) {
      Slot sl = load_slot(tb, cfg.slot);
      if (cfg.lexnode != kNoLex && cfg.lexnode >= sl.nodes) b = 1;
    }
    bad = b;
    overflow = 0;
    nA = 0;
  }
  if (tid < 8) {
    A[tid] = 0;
    uint32_t iw = 0;
    for (int j = 0; j < 32; ++j) {
      int t = tid * 32 + j;
      if (t < tb.T && (tb.term_info[t] & 1u)) iw |= 1u << j;
    }
    I[tid] = iw;
  }
  for (int w = tid; w < tb.W; w += kBlock) mrow[w] = 0u;
  __syncthreads();
  const uint32_t depth = cfg.stk_depth;
  const uint32_t lo = depth > (uint32_t)kStackWin ? depth - kStackWin : 0;
  if (!bad) {
    for (uint32_t i = tid; i < depth; i += kBlock) {
      uint16_t s = pool[cfg.stk_off + i];
      if (s >= tb.NS) bad = 1;
      if (i >= lo) win[i - lo] = s;
    }
  }
  __syncthreads();
  if (bad) {
    if (tid == 0) {
      hdr->valid = 0;
      hdr->status = GRID_ROW_BAD_CONFIG;
      hdr->eos_ok = 0;
      if (eos_out) eos_out[row] = 0;
    }
    return;
  }
  BaseStack bs{pool + cfg.stk_off, win, depth, lo};
  Post* post = row_post(rw);
  uint16_t* my = scratch[tid];

  // A(sigma) and the stack after each allowed terminal's shift
  for (int t = tid; t < tb.T; t += kBlock) {
    uint32_t k = depth;
    int m = 0;
    int r = sim_shift(tb, bs, k, m, my, kPostCap, t);
    Post p;
    p.k = (uint16_t)k;
    p.m = (uint8_t)m;
    p.ok = r == 1;
    for (int j = 0; j < kPostCap; ++j) p.ov[j] = j < m ? my[j] : 0;
    if (r == 1) {
      if (k > 0xFFFF) overflow = 1;
      atomicOr(&A[t >> 5], 1u << (t & 31));
    }
    if (r < 0) overflow = 1;
    post[t] = p;
  }
  for (int i = tid; i < 256 * 8; i += kBlock) A2s[i] = 0;
  __syncthreads();
  if (tid == 0) {
    int n = 0;
    for (int t = 0; t < tb.T; ++t)
      if ((A[t >> 5] >> (t & 31)) & 1u) alist[n++] = (uint8_t)t;
    nA = n;
  }
  __syncthreads();
  // allowed set after each first shift: A(sigma'_t) for t in A(sigma)
  const int pairs = nA * tb.T;
  for (int idx = tid; idx < pairs; idx += kBlock) {
    int t = alist[idx / tb.T], x = idx % tb.T;
    const Post& p = post[t];
    int r = sim_test(tb, bs, p.k, p.m, p.ov, my, x);
    if (r == 1) atomicOr(&A2s[t * 8 + (x >> 5)], 1u << (x & 31));
    if (r < 0) overflow = 1;
  }
  __syncthreads();
  uint32_t* a2 = row_a2(rw, tb.T);
  for (int i = tid; i < tb.T * 8; i += kBlock) a2[i] = A2s[i];

  const Slot sl = load_slot(tb, cfg.slot);
  // trailing-lexeme code per DFA state under A(sigma): bit 15 = viable
  // through an unrestricted terminal, bits 0..7 = categories whose lexicon
  // prefix test decides
  uint16_t* vend = row_vend(rw, tb.T);
  for (int q = tid; q < tb.S; q += kBlock) {
    uint32_t code = 0;
    for (int w = 0; w < 8; ++w) {
      uint32_t bits = tb.live[(size_t)q * 8 + w] & (A[w] | I[w]);
      while (bits) {
        int t = w * 32 + __ffs(bits) - 1;
        bits &= bits - 1;
        uint32_t c;
        if (restricted_cat(sl, tb.term_info[t], c)) code |= 1u << c;
        else code |= 0x8000u;
      }
    }
    vend[q] = (uint16_t)code;
  }
  // end-of-sequence gate (mid-lexeme aware)
  if (tid == 0) {
    int ok = 0;
    if (cfg.flags & 1u) {
      ok = sim_test(tb, bs, depth, 0, my, my + kPostCap, tb.T) == 2;
    } else {
      int winner = -1;
      for (uint32_t j = tb.acc_off[cfg.q]; j < tb.acc_off[cfg.q + 1]; ++j) {
        int t = tb.acc_list[j];
        uint32_t ti = tb.term_info[t];
        bool allowed = (ti & 1u) || ((A[t >> 5] >> (t & 31)) & 1u);
        uint32_t c;
        bool lexok = !restricted_cat(sl, ti, c) ||
                     ((lex_flags_of(tb, sl, cfg.lexnode) >> (8 + c)) & 1u);
        if (allowed && lexok) {
          winner = t;
          break;
        }
      }
      if (winner >= 0) {
        if (tb.term_info[winner] & 1u) {
          ok = sim_test(tb, bs, depth, 0, my, my + kPostCap, tb.T) == 2;
        } else {
          const Post& p = post[winner];
          ok = sim_test(tb, bs, p.k, p.m, p.ov, my + kPostCap, tb.T) == 2;
        }
      }
    }
    hdr->eos_ok = (uint32_t)ok;
    if (eos_out) eos_out[row] = (uint8_t)ok;
    if (ok && tb.eos_id >= 0) mrow[tb.eos_id >> 5] |= 1u << (tb.eos_id & 31);
  }
  __syncthreads();
  if (tid < 8) hdr->A[tid] = A[tid];
  if (tid == 0) {
    hdr->status = overflow ? GRID_ROW_OVERFLOW : GRID_ROW_OK;
    hdr->valid = kRowValid;
  }
}

// -------------------------------------------------------------------- walk
struct LaneCtx {
  const Tables& tb;
  const BaseStack& bs;
  const Slot& sl;
  const uint32_t* A;       // LDS
  const uint16_t* vend;    // LDS
  const uint32_t* a2;      // global, this row
  const Post* post;        // global, this row
  uint16_t* ov;            // LDS, this lane
  uint16_t* tmp;           // LDS, this lane
  int mode;                // 0: stack sigma; 1: after first shift t1; 2: own overlay
  int t1;
  uint32_t k;
  int m;
  int err;

  __device__ bool in_A(int x) {
    if (mode == 0) return (A[x >> 5] >> (x & 31)) & 1u;
    if (mode == 1) return (a2[t1 * 8 + (x >> 5)] >> (x & 31)) & 1u;
    int r = sim_test(tb, bs, k, m, ov, tmp, x);
    if (r < 0) err = 1;
    return r == 1;
  }
  __device__ bool viable_now(int q, uint32_t lex) {
    if (mode == 0) {
      uint32_t code = vend[q];
      if (code & 0x8000u) return true;
      return (lex_flags_of(tb, sl, lex) & code & 0xFFu) != 0;
    }
    uint32_t lf = lex_flags_of(tb, sl, lex);
    for (int w = 0; w < 8; ++w) {
      uint32_t bits = tb.live[(size_t)q * 8 + w];
      while (bits) {
        int t = w * 32 + __ffs(bits) - 1;
        bits &= bits - 1;
        uint32_t ti = tb.term_info[t], c;
        if (restricted_cat(sl, ti, c) && !((lf >> c) & 1u)) continue;
        if ((ti & 1u) || in_A(t)) return true;
      }
    }
    return false;
  }
  // emit the pending lexeme in state q; false = reject
  __device__ bool emit(int q, uint32_t lex) {
    uint32_t a0 = tb.acc_off[q], a1 = tb.acc_off[q + 1];
    if (a0 == a1) return false;
    uint32_t lf = lex_flags_of(tb, sl, lex);
    int winner = -1;
    for (uint32_t j = a0; j < a1; ++j) {
      int t = tb.acc_list[j];
      uint32_t ti = tb.term_info[t], c;
      if (restricted_cat(sl, ti, c) && !((lf >> (8 + c)) & 1u)) continue;
      if ((ti & 1u) || in_A(t)) {
        winner = t;
        break;
      }
    }
    if (winner < 0) return false;
    if (tb.term_info[winner] & 1u) return true;  // ignored: the stack is unchanged
    if (mode == 0) {
      mode = 1;
      t1 = winner;
      return true;
    }
    if (mode == 1) {
      const Post& p = post[t1];
      if (p.k == 0 || p.k > bs.depth || p.m > kPostCap) {  // workspace not from a prologue
        err = 1;
        return false;
      }
      k = p.k;
      m = p.m;
      for (int j = 0; j < m; ++j) {
        ov[j] = p.ov[j];
        if (ov[j] >= tb.NS) {
          err = 1;
          return false;
        }
      }
      mode = 2;
    }
    int r = sim_shift(tb, bs, k, m, ov, kOvCap, winner);
    if (r < 0) err = 1;
    return r == 1;
  }
};

__global__ __launch_bounds__(kBlock) void walk_kernel(Tables tb, const grid_config* __restrict__ cfgs,
                                                      const uint16_t* __restrict__ pool,
                                                      uint32_t* __restrict__ mask,
                                                      uint8_t* __restrict__ ws, size_t rbytes) {
  extern __shared__ uint8_t lds[];
  const int row = blockIdx.y;
  const int tid = threadIdx.x;
  uint8_t* rw = ws + (size_t)row * rbytes;
  RowHeader* hdr = (RowHeader*)rw;
  if (hdr->valid != kRowValid) return;
  const grid_config cfg = cfgs[row];

  uint32_t* A = (uint32_t*)lds;                                  // 8 words
  uint16_t* win = (uint16_t*)(lds + 32);                         // kStackWin
  uint16_t* vend = win + kStackWin;                              // S (padded)
  uint16_t* lanes = vend + ((tb.S + 7) & ~7);                    // kBlock * kLaneWords
  if (tid < 8) A[tid] = hdr->A[tid];
  const uint32_t depth = cfg.stk_depth;
  const uint32_t lo = depth > (uint32_t)kStackWin ? depth - kStackWin : 0;
  for (uint32_t i = lo + tid; i < depth; i += kBlock) win[i - lo] = pool[cfg.stk_off + i];
  const uint16_t* vsrc = row_vend(rw, tb.T);
  for (int q = tid; q < tb.S; q += kBlock) vend[q] = vsrc[q];
  __syncthreads();

  const BaseStack bs{pool + cfg.stk_off, win, depth, lo};
  const Slot sl = load_slot(tb, cfg.slot);
  const uint32_t* a2 = row_a2(rw, tb.T);
  const Post* post = row_post(rw);
  uint16_t* mine = lanes + (size_t)tid * kLaneWords;
  uint32_t* mrow = mask + (size_t)row * tb.W;
  int any_err = 0;

  const int u_end = min(tb.U, (int)(blockIdx.x + 1) * kSpellPerBlock);
  for (int u = blockIdx.x * kSpellPerBlock + tid; u < u_end; u += kBlock) {
    LaneCtx lc{tb, bs, sl, A, vend, a2, post, mine, mine + kOvCap, 0, -1, 0, 0, 0};
    uint32_t i = tb.spell_off[u];
    const uint32_t end = tb.spell_off[u + 1];
    int q = cfg.q;
    uint32_t lex = cfg.lexnode;
    bool ok = true;
    for (; i < end; ++i) {
      const uint32_t b = tb.spell_bytes[i];
      const uint32_t c = tb.bclass[b];
      const int nq = tb.dfa[(size_t)q * tb.C + c];
      if (nq != kDead) {
        q = nq;
        lex = lex_child(tb, sl, lex, b);
      } else {
        if (!lc.emit(q, lex)) {
          ok = false;
          break;
        }
        q = tb.dfa[(size_t)kStart * tb.C + c];
        if (q == kDead) {
          ok = false;
          break;
        }
        lex = lex_child(tb, sl, 0u, b);
      }
      if (!lc.viable_now(q, lex)) {
        ok = false;
        break;
      }
    }
    any_err |= lc.err;
    if (ok) {
      for (uint32_t j = tb.alias_off[u]; j < tb.alias_off[u + 1]; ++j) {
        const int id = tb.alias_ids[j];
        atomicOr(&mrow[id >> 5], 1u << (id & 31));
      }
    }
  }
  if (any_err) atomicOr(&hdr->status, GRID_ROW_OVERFLOW);
}

// ---------------------------------------------------------------- finalize
__global__ __launch_bounds__(kBlock) void finalize_kernel(Tables tb, const uint32_t* __restrict__ mask,
                                                          const uint8_t* __restrict__ ws, size_t rbytes,
                                                          int32_t* __restrict__ status) {
  const int row = blockIdx.x;
  const RowHeader* hdr = (const RowHeader*)(ws + (size_t)row * rbytes);
  __shared__ uint32_t any;
  if (threadIdx.x == 0) any = 0;
  __syncthreads();
  const uint32_t* mrow = mask + (size_t)row * tb.W;
  uint32_t acc = 0;
  for (int w = threadIdx.x; w < tb.W; w += kBlock) acc |= mrow[w];
  if (acc) atomicOr(&any, 1u);
  __syncthreads();
  if (threadIdx.x == 0) {
    int32_t st = hdr->status;
    if (hdr->valid == kRowValid && !any && !hdr->eos_ok) st |= GRID_ROW_EMPTY;
    status[row] = st;
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

}  // namespace

int grid::overlay_capacity() { return kOvCap; }

extern "C" size_t grid_mask_workspace_bytes(const grid_compiled* g, int32_t B) {
  if (!g || B <= 0) return 0;
  return row_bytes(g->parser.T, g->dfa.S) * (size_t)B;
}

extern "C" int grid_mask_phases(const grid_compiled* g, int32_t B, const grid_config* cfg_dev,
                                const uint16_t* stack_pool_dev, uint32_t* mask_dev, uint8_t* eos_dev,
                                int32_t* status_dev, void* workspace_dev, size_t workspace_bytes,
                                uint32_t phases, void* stream) {
  clear_error();
  if (phases & ~GRID_PHASE_ALL) return fail(GRID_E_ARG, "grid_mask: unknown phase bits");
  if (!g || B <= 0 || B > 65535 || !cfg_dev || !stack_pool_dev || !mask_dev || !workspace_dev)
    return fail(GRID_E_ARG, "grid_mask: null pointer or batch size out of range");
  const size_t rb = row_bytes(g->parser.T, g->dfa.S);
  if (workspace_bytes < rb * (size_t)B) return fail(GRID_E_ARG, "grid_mask: workspace too small");
  static const int needed[] = {GRID_ART_DFA_CLASS,  GRID_ART_BYTE_CLASS, GRID_ART_DFA_ACCEPT_OFF,
                               GRID_ART_DFA_ACCEPT_LIST, GRID_ART_DFA_LIVE, GRID_ART_ACTION,
                               GRID_ART_GOTO,       GRID_ART_PROD,       GRID_ART_TERM_INFO,
                               GRID_ART_SPELL_OFF,  GRID_ART_SPELL_BYTES, GRID_ART_ALIAS_OFF,
                               GRID_ART_ALIAS_IDS,  GRID_ART_LEX_FLAGS,  GRID_ART_LEX_HASH,
                               GRID_ART_LEX_SLOTS};
  for (int w : needed)
    if (!bound(g, w)) return fail(GRID_E_UNBOUND, "grid_mask: artifact " + std::to_string(w) + " is not bound");
  Tables tb;
  tb.dfa = (const uint16_t*)g->dev[GRID_ART_DFA_CLASS];
  tb.bclass = (const uint8_t*)g->dev[GRID_ART_BYTE_CLASS];
  tb.acc_off = (const uint32_t*)g->dev[GRID_ART_DFA_ACCEPT_OFF];
  tb.acc_list = (const uint8_t*)g->dev[GRID_ART_DFA_ACCEPT_LIST];
  tb.live = (const uint32_t*)g->dev[GRID_ART_DFA_LIVE];
  tb.action = (const uint16_t*)g->dev[GRID_ART_ACTION];
  tb.go = (const uint16_t*)g->dev[GRID_ART_GOTO];
  tb.prod = (const uint32_t*)g->dev[GRID_ART_PROD];
  tb.term_info = (const uint32_t*)g->dev[GRID_ART_TERM_INFO];
  tb.spell_off = (const uint32_t*)g->dev[GRID_ART_SPELL_OFF];
  tb.spell_bytes = (const uint8_t*)g->dev[GRID_ART_SPELL_BYTES];
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
  tb.U = (int)g->vocab.spell_off.size() - 1;
  tb.V = g->vocab.V;
  tb.W = (g->vocab.V + 31) / 32;
  tb.n_slots = g->lex.n_slots;
  tb.eos_id = g->vocab.eos_id;
  if (tb.S > 8192) return fail(GRID_E_CAPACITY, "grid_mask: more than 8192 DFA states");
  hipStream_t s = (hipStream_t)stream;
  uint8_t* ws = (uint8_t*)workspace_dev;
  if (phases & GRID_PHASE_PROLOGUE)
    hipLaunchKernelGGL(prologue_kernel, dim3(B), dim3(kBlock), 0, s, tb, cfg_dev, stack_pool_dev, mask_dev,
                       eos_dev, ws, rb);
  if ((phases & GRID_PHASE_WALK) && tb.U > 0) {
    const size_t lds = 32 + kStackWin * 2 + (size_t)((tb.S + 7) & ~7) * 2 + (size_t)kBlock * kLaneWords * 2;
    dim3 grid((tb.U + kSpellPerBlock - 1) / kSpellPerBlock, B);
    hipLaunchKernelGGL(walk_kernel, grid, dim3(kBlock), lds, s, tb, cfg_dev, stack_pool_dev, mask_dev, ws, rb);
  }
  if ((phases & GRID_PHASE_FINALIZE) && status_dev)
    hipLaunchKernelGGL(finalize_kernel, dim3(B), dim3(kBlock), 0, s, tb, mask_dev, ws, rb, status_dev);
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
