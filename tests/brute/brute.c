/*
 * brute.c -- exhaustive checker for the oracle on two tiny grammars.
 *
 * Test infrastructure.  For each grammar a hand-written lexer and a
 * hand-written pushdown recognizer decide membership in L (no regex engine, no
 * Earley, no tables).  Every byte string over a small alphabet up to length K
 * is enumerated; a string is a viable prefix iff some extension of total length
 * <= K is a member (the definition of Prefix(L), Proposition 2, restricted to a
 * length bound).  For query strings (length <= KQ) the checker reports
 * membership, bounded viability, and whether the bounded answer is exact:
 * it is when a completion was found, when the recognizer already rejected an
 * emitted lexeme (rejection is monotone), or when the string plus the
 * grammar's longest shortest-completion still fits in K.
 *
 * Grammar 0: expression grammar (E -> E+T|T, T -> T*F|F, F -> (E)|NUM|ID),
 *            alphabet {1 a + * ( ) space}.
 * Grammar 1: keyword/identifier/lexicon grammar
 *            S -> cols opt "g" TBL ; opt -> eps | "!" ; cols -> COL | cols "," COL
 *            with TBL = {b, ba, bab}, COL = {a, ab, g, bb}, keyword "g"
 *            (priority above the identifiers), alphabet {a b g , ! space}.
 */
#include <stdint.h>
#include <string.h>

enum { REJ = 0, PENDING = 1 };

/* ---------------------------------------------------------------- grammar 0 */
static const char ALPHA0[] = "1a+*() ";

static int is_digit(char c) { return c >= '0' && c <= '9'; }
static int is_lower(char c) { return c >= 'a' && c <= 'z'; }

/* Runs the recognizer over s; returns REJ or PENDING.  *member is set when
 * the whole string (with the pending lexeme finalized) is a sentence; *open
 * receives the parenthesis depth. */
static int expr_run(const char* s, int n, int* member, int* open) {
  int expect_operand = 1, depth = 0, i = 0;
  *member = 0;
  *open = 0;
  while (i < n) {
    char c = s[i];
    int j = i + 1, kind;  /* 0 operand, 1 plus/star, 2 lparen, 3 rparen, 4 ws */
    if (is_digit(c)) {
      while (j < n && is_digit(s[j])) ++j;
      kind = 0;
    } else if (is_lower(c)) {
      while (j < n && (is_lower(s[j]) || is_digit(s[j]))) ++j;
      kind = 0;
    } else if (c == '+' || c == '*') {
      kind = 1;
    } else if (c == '(') {
      kind = 2;
    } else if (c == ')') {
      kind = 3;
    } else if (c == ' ') {
      while (j < n && s[j] == ' ') ++j;
      kind = 4;
    } else {
      return REJ;
    }
    /* A lexeme that reaches the end of the string is still pending; it is
     * emitted here too, which is what finalization at end of input does.  A
     * pending operand can only grow into an operand, so checking it now is
     * monotone-safe for the rejection test as well. */
    if (kind == 4) {
      /* ignored */
    } else if (expect_operand) {
      if (kind == 0) expect_operand = 0;
      else if (kind == 2) ++depth;
      else return REJ;
    } else {
      if (kind == 1) expect_operand = 1;
      else if (kind == 3 && depth > 0) --depth;
      else return REJ;
    }
    i = j;
  }
  *member = (!expect_operand && depth == 0);
  *open = depth;
  return PENDING;
}

/* ---------------------------------------------------------------- grammar 1 */
static const char ALPHA1[] = "abg,! ";

static int in_list(const char* w, int n, const char* const* list) {
  for (int k = 0; list[k]; ++k)
    if ((int)strlen(list[k]) == n && memcmp(list[k], w, (size_t)n) == 0) return 1;
  return 0;
}

static const char* const TBL_WORDS[] = {"b", "ba", "bab", 0};
static const char* const COL_WORDS[] = {"a", "ab", "g", "bb", 0};

/* parser states: 0 expect COL; 1 after COL (expect , ! g); 2 after ','
 * (expect COL); 3 after '!' (expect g); 4 after g (expect TBL); 5 done */
static int lexi_run(const char* s, int n, int* member, int* unused) {
  int st = 0, i = 0;
  (void)unused;
  *member = 0;
  while (i < n) {
    char c = s[i];
    int j = i + 1;
    if (is_lower(c)) {
      while (j < n && is_lower(s[j])) ++j;
      int len = j - i;
      int pending = (j == n);
      /* candidates in priority order: KG, TBL, COL */
      int kg = (len == 1 && c == 'g');
      int tb = in_list(s + i, len, TBL_WORDS);
      int cl = in_list(s + i, len, COL_WORDS);
      int next = -1;
      if (kg && (st == 1 || st == 3)) next = 4;
      else if (tb && st == 4) next = 5;
      else if (cl && (st == 0 || st == 2)) next = 1;
      if (next < 0) {
        if (pending) return PENDING; /* the lexeme may still grow */
        return REJ;
      }
      if (pending) {
        /* finalization at end of input picks this winner */
        st = next;
        *member = (st == 5);
        return PENDING;
      }
      st = next;
    } else if (c == ',') {
      if (st != 1) return REJ;
      st = 2;
    } else if (c == '!') {
      if (st != 1) return REJ;
      st = 3;
    } else if (c == ' ') {
      while (j < n && s[j] == ' ') ++j;
    } else {
      return REJ;
    }
    i = j;
  }
  *member = (st == 5);
  return PENDING;
}

/* --------------------------------------------------------------- enumeration */
typedef int (*run_fn)(const char*, int, int*, int*);

static run_fn RUN;
static const char* ALPHA;
static int A, K, KQ, BOUND_CONST;
static uint8_t *OUT_M, *OUT_V, *OUT_D;
static int64_t BASE[32]; /* offset of length-L block in the outputs */
static char BUF[64];

static int dfs(int len, int64_t code) {
  int member = 0, open = 0;
  int st = RUN(BUF, len, &member, &open);
  int viable = member;
  if (st == REJ) viable = 0;
  /* a rejected string's extensions are rejected too; they are still walked up
   * to the query length so that their entries get recorded */
  if ((st != REJ || len < KQ) && len < K) {
    for (int c = 0; c < A && (len < KQ || !viable); ++c) {
      BUF[len] = ALPHA[c];
      viable |= dfs(len + 1, code * A + c);
    }
  }
  if (len <= KQ) {
    int64_t idx = BASE[len] + code;
    OUT_M[idx] = (uint8_t)member;
    OUT_V[idx] = (uint8_t)viable;
    int bound = BOUND_CONST >= 0 ? BOUND_CONST : open + 1;
    OUT_D[idx] = (uint8_t)(viable || st == REJ || len + bound <= K);
  }
  return viable;
}

/* Outputs are indexed by length block (lengths 0..kq, block L holds A^L
 * entries) and, within a block, by the base-A code of the string (first
 * character most significant, alphabet order as returned by brute_alphabet). */
int brute_run(int grammar, int k, int kq, uint8_t* out_member, uint8_t* out_viable,
              uint8_t* out_decided) {
  if (grammar == 0) {
    RUN = expr_run;
    ALPHA = ALPHA0;
    BOUND_CONST = -1; /* completion needs one operand plus the open parens */
  } else {
    RUN = lexi_run;
    ALPHA = ALPHA1;
    BOUND_CONST = 6; /* e.g. a pending "b" at the start: "b g b" */
  }
  A = (int)strlen(ALPHA);
  K = k;
  KQ = kq;
  if (K > 60 || KQ > K) return -1;
  OUT_M = out_member;
  OUT_V = out_viable;
  OUT_D = out_decided;
  int64_t off = 0, p = 1;
  for (int L = 0; L <= KQ; ++L) {
    BASE[L] = off;
    off += p;
    p *= A;
  }
  dfs(0, 0);
  return 0;
}

const char* brute_alphabet(int grammar) { return grammar == 0 ? ALPHA0 : ALPHA1; }

int brute_member(int grammar, const char* s, int n) {
  int m = 0, o = 0;
  int st = (grammar == 0 ? expr_run : lexi_run)(s, n, &m, &o);
  return st == REJ ? 0 : m;
}
