"""Pins of the CPU oracle against things other than itself.

* an exhaustive brute-force enumeration with hand-written recognizers
  (tests/brute/brute.c) on two tiny grammars: viability (Definition 2),
  membership (end of sequence), and the mask of Definition 4;
* the first worked example of section 7.1 (tests/golden/worked_example_1.json);
* textbook allowed-terminal sets of the expression grammar's LR automaton;
* Proposition 2 (the first-step mask is nonempty), monotone rejection under
  extension (section 4.1), alias equality (section 2, alias classes),
  special tokens and padding bits;
* the role projection (section 2, L2): dropped verbs are outside the language;
* checkpoint mode equals from-scratch mode (on the workloads and on random
  grammars with keywords and lexicon categories);
* on random grammars with context-free lexing, viability, membership and the
  mask equal those of a plain CYK-style check that decides Prefix(L) exactly.
"""

import itertools
import json
from pathlib import Path

import numpy as np
import pytest

from workloads import grammar_text, make_workload

GOLDEN = Path(__file__).resolve().parent / "golden"

LEXI_LEXICON = {"TBL": ["b", "ba", "bab"], "COL": ["a", "ab", "g", "bb"]}


def _brute_table(brute, grammar, K, KQ):
    alpha = brute.brute_alphabet(grammar)
    A = len(alpha)
    n = sum(A ** L for L in range(KQ + 1))
    m = np.zeros(n, np.uint8)
    v = np.zeros(n, np.uint8)
    d = np.zeros(n, np.uint8)
    assert brute.brute_run(grammar, K, KQ, m.ctypes.data, v.ctypes.data, d.ctypes.data) == 0
    table = {}
    idx = 0
    for L in range(KQ + 1):
        for combo in itertools.product(alpha, repeat=L):
            table[bytes(combo)] = (bool(m[idx]), bool(v[idx]), bool(d[idx]))
            idx += 1
    return table


def _oracle_for(oracle_mod, name, vocab=None):
    lex = LEXI_LEXICON if name == "lexi" else None
    if vocab is None:
        vocab = [b"x"]
    return oracle_mod.Oracle(grammar_text(name), (), lex, vocab)


@pytest.mark.parametrize("name,gid,K,KQ", [("expr", 0, 9, 6), ("lexi", 1, 10, 6)])
def test_oracle_matches_brute_force(oracle_mod, brute, name, gid, K, KQ):
    table = _brute_table(brute, gid, K, KQ)
    o = _oracle_for(oracle_mod, name)
    undecided = 0
    checked = 0
    n_viable = n_member = 0
    for s, (mem, via, dec) in table.items():
        assert o.member(s) == mem, (s, "membership")
        n_member += mem
        if not dec:
            undecided += 1
            continue
        checked += 1
        n_viable += via
        assert o.viable(s) == via, (s, "viability")
    # the enumeration must actually decide most strings and contain both answers
    assert checked > 0.9 * len(table)
    assert n_member > 20 and n_viable > 200 and checked - n_viable > 200


@pytest.mark.parametrize("name,gid,K,KQ", [("expr", 0, 9, 6), ("lexi", 1, 10, 6)])
def test_oracle_mask_matches_brute_force(oracle_mod, brute, name, gid, K, KQ):
    table = _brute_table(brute, gid, K, KQ)
    alpha = brute.brute_alphabet(gid)
    vocab = [bytes([c]) for c in alpha] + [bytes(p) for p in itertools.product(alpha, repeat=2)]
    vocab.append(b"")  # an end-of-sequence special with empty spelling
    eos = len(vocab) - 1
    lex = LEXI_LEXICON if name == "lexi" else None
    o = oracle_mod.Oracle(grammar_text(name), (), lex, vocab, [eos], eos)
    prefixes = [bytes(p) for L in range(4) for p in itertools.product(alpha, repeat=L)]
    rng = np.random.default_rng(7)
    prefixes += [rng.choice(np.frombuffer(alpha, np.uint8), size=4).tobytes() for _ in range(150)]
    compared = 0
    for w in prefixes:
        for mode in (0, 1):
            words, eos_ok = o.mask(w, mode=mode, nthreads=1)
            assert eos_ok == table[w][0], (w, mode)
            for t, sp in enumerate(vocab[:-1]):
                mem, via, dec = table[w + sp]
                bit = (int(words[t >> 5]) >> (t & 31)) & 1
                if dec:
                    compared += 1
                    assert bit == via, (w, sp, mode)
            assert ((int(words[eos >> 5]) >> (eos & 31)) & 1) == eos_ok
    assert compared > 10000


def test_worked_example_section_7_1(oracle_mod):
    fx = json.loads((GOLDEN / "worked_example_1.json").read_text())
    spells = sorted({s for c in fx["cases"] for k in ("allowed", "blocked") for s in c.get(k, [])})
    vocab = [s.encode() for s in spells] + [b""]
    eos = len(vocab) - 1
    o = oracle_mod.Oracle(grammar_text(fx["grammar"]), fx["drop"], fx["lexicon"], vocab, [eos], eos)
    for c in fx["cases"]:
        w = c["prefix"].encode()
        for mode in (0, 1):
            words, eos_ok = o.mask(w, mode=mode)
            bits = {spells[t]: (int(words[t >> 5]) >> (t & 31)) & 1 for t in range(len(spells))}
            for s in c.get("allowed", []):
                assert bits[s] == 1, (c["prefix"], s)
            for s in c.get("blocked", []):
                assert bits[s] == 0, (c["prefix"], s)
            if "eos" in c:
                assert eos_ok == int(c["eos"]), c["prefix"]
    # the statement head still admits the kept verb
    assert o.viable(b"select") and o.viable(b"sel")


def test_textbook_allowed_sets_expr(oracle_mod):
    """Allowed next terminals of the expression grammar, derivable by hand from
    its LR automaton: after '(' an operand is needed; after a complete operand
    at depth 0 only an operator (or the end) may follow; inside parens ')' too."""
    o = _oracle_for(oracle_mod, "expr")
    cases = {
        b"": {"LPAREN", "NUM", "ID"},
        b"(": {"LPAREN", "NUM", "ID"},
        b"1 ": {"PLUS", "STAR"},
        b"(1 ": {"PLUS", "STAR", "RPAREN"},
        b"1+": {"PLUS", "STAR"},             # '+' is still pending
        b"1+ ": {"LPAREN", "NUM", "ID"},
        b"(a)": {"PLUS", "STAR", "RPAREN"},  # ")" is still pending
        b"(a) ": {"PLUS", "STAR"},
        b"a*(b+c)* ": {"LPAREN", "NUM", "ID"},
    }
    for w, want in cases.items():
        ok, got = o.allowed(w)
        assert ok and got == want, (w, got)
    assert o.member(b"1") and o.member(b"(a1 + 22) * b ") and not o.member(b"(1")
    assert not o.viable(b"1a") and not o.viable(b")")  # NUM then ID; a stray ')'


def test_contextual_resolution_lexi(oracle_mod):
    """'g' is a keyword where the keyword is viable and a column where only a
    column is (section 2, contextual resolution)."""
    o = _oracle_for(oracle_mod, "lexi")
    assert o.member(b"g g b")        # column g, keyword g, table b
    assert o.member(b"a,g g ba")
    assert not o.viable(b"a gb")     # 'gb' is one lexeme and no word
    assert not o.viable(b"ab g bb")  # bb is a column, not a table
    assert o.viable(b"a g ba") and not o.viable(b"a g bax")
    assert o.member(b"a ! g bab ")


def test_prefix_semantics_first_step_nonempty(oracle_mod):
    """Proposition 2: with prefix semantics the first mask is not empty even
    though no one-token string is a sentence."""
    for k in (1, 2, 3):
        wl = make_workload(k, rows=1)
        o = oracle_mod.from_workload(wl)
        words, eos_ok = o.mask(b"", mode=1)
        assert int(np.unpackbits(words.view(np.uint8)).sum()) > 0
        assert eos_ok == 0


def test_modes_agree_and_invariants_expr(oracle_mod):
    wl = make_workload(1, rows=24)
    o = oracle_mod.from_workload(wl)
    V = wl.V
    for w in wl.prefixes:
        a, ea = o.mask(w, mode=0)
        b, eb = o.mask(w, mode=1)
        assert np.array_equal(a, b) and ea == eb
        bits = [(int(a[t >> 5]) >> (t & 31)) & 1 for t in range(V)]
        spell = wl.vocab
        # alias classes: equal spellings, equal bits
        by = {}
        for t in range(V):
            by.setdefault(spell[t], set()).add(bits[t])
        assert all(len(s) == 1 for s in by.values())
        # monotone rejection: a blocked spelling blocks its extensions
        blocked = {spell[t] for t in range(V) if not bits[t]}
        for t in range(V):
            if bits[t]:
                for k in range(1, len(spell[t])):
                    assert spell[t][:k] not in blocked, (w, spell[t])
        # byte completeness + viable prefix => some byte is allowed
        assert o.viable(w)
        assert any(bits[:256])


@pytest.mark.parametrize("k,n_rows,n_rand", [(2, 8, 1500), (3, 16, 1500), (4, 12, 300)])
def test_modes_agree_on_sql_workloads(oracle_mod, k, n_rows, n_rand):
    """From-scratch mode (every token re-lexes and re-parses the whole
    extended prefix, the plain reading of Definition 4) equals checkpoint mode
    (the prefix parsed once) on the SQL grammars the GPU parity tests use:
    seeded rows of workloads 2 and 3, and one row of every (position, depth)
    cell of the 16,000-token workload (the longest and most deeply nested
    prefixes), each on a seeded token subset of random ids plus ids the
    checkpoint mask allows, so both verdicts are exercised."""
    wl = make_workload(k)
    o = oracle_mod.from_workload(wl)
    rng = np.random.default_rng(6100 + k)
    if k == 4:
        rows = [c * wl.batch + int(rng.integers(wl.batch)) for c in range(len(wl.prefixes) // wl.batch)]
    else:
        rows = sorted(rng.choice(len(wl.prefixes), n_rows, replace=False).tolist())
    n_allowed = 0
    for j in rows:
        w = wl.prefixes[j]
        full, e1 = o.mask(w, mode=1)
        bits = np.unpackbits(full.view(np.uint8), bitorder="little")[:wl.V]
        allowed = np.flatnonzero(bits)
        pick = rng.choice(allowed, min(len(allowed), n_rand), replace=False) if len(allowed) else allowed
        toks = np.unique(np.concatenate([rng.choice(wl.V, n_rand, replace=False), pick])).astype(np.int32)
        b0, e0 = o.mask(w, mode=0, tokens=toks)
        b1, e1b = o.mask(w, mode=1, tokens=toks)
        assert np.array_equal(b0, b1), (k, j, toks[np.flatnonzero(b0 != b1)][:8].tolist())
        assert np.array_equal(b1, bits[toks]), (k, j)
        assert e0 == e1 == e1b, (k, j)
        n_allowed += int(b0.sum())
    assert n_allowed > 0


def test_generated_sentences_are_members(oracle_mod):
    import random
    from workloads import sentences as sen
    for k in (1, 2, 3):
        wl = make_workload(k, rows=2)
        o = oracle_mod.from_workload(wl)
        r = random.Random(17)
        for _ in range(20):
            if k == 1:
                s = sen.gen_expr(r)
            elif k == 2:
                s = sen.SelectSubsetGen(r, wl.meta["schema"]).sentence()
            else:
                s = sen.DmlQueryGen(r, wl.meta["schema"]).sentence()
            b = s.encode()
            assert o.member(b), s
            cut = r.randint(0, len(b))
            assert o.viable(b[:cut]), b[:cut]


def test_workload_prefixes_viable(oracle_mod):
    for k in (1, 2, 3):
        wl = make_workload(k)
        o = oracle_mod.from_workload(wl)
        for w in wl.prefixes:
            assert o.viable(w), (k, w)


def test_role_projection_blocks_verbs(oracle_mod):
    wl = make_workload(3, rows=1)
    o = oracle_mod.from_workload(wl)
    for verb in (b"insert", b"update", b"delete", b"INSERT", b"Delete"):
        assert not o.viable(verb)
        assert not o.viable(b"  " + verb)
    assert o.viable(b"select") and o.viable(b"WITH")
    full = oracle_mod.Oracle(grammar_text("sql_dml"), (), wl.lexicons[0], wl.vocab)
    assert full.viable(b"insert into ")


def test_specials_and_padding_zero(oracle_mod):
    wl = make_workload(2, rows=2)
    o = oracle_mod.from_workload(wl)
    words, eos_ok = o.mask(wl.prefixes[0], mode=1)
    V = wl.V
    for t in wl.specials:
        if t != wl.eos_id:
            assert (int(words[t >> 5]) >> (t & 31)) & 1 == 0
    assert ((int(words[wl.eos_id >> 5]) >> (wl.eos_id & 31)) & 1) == eos_ok
    pad = int(words[-1]) >> (V & 31) if V & 31 else 0
    assert pad == 0


def test_eos_after_complete_statement(oracle_mod):
    wl = make_workload(3, rows=1)
    o = oracle_mod.from_workload(wl)
    s = wl.meta["schema"]
    sent = f"select {s.columns[0][0]} from {s.tables[0]} ;".encode()
    _, eos_ok = o.mask(sent, mode=1, tokens=[0])
    assert eos_ok == 1
    _, eos_ok = o.mask(sent[:-1], mode=1, tokens=[0])
    assert eos_ok == 0
    _, eos_ok = o.mask(sent + b" \n", mode=1, tokens=[0])
    assert eos_ok == 1


def test_error_paths(oracle_mod):
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.Grammar(grammar_text("crud"), ["select", "insert", "update", "delete"])
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.Grammar(grammar_text("crud"), ["nosuchlabel"])
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.Grammar("start S\ntoken A /[a-/\nS : A ;\n")
    with pytest.raises(oracle_mod.OracleError):
        oracle_mod.Grammar("start S\ntoken A \"a\"\nS : A B ;\n")


def test_priority_decides_between_viable_candidates(oracle_mod):
    """Contextual resolution picks the highest-priority viable candidate
    (section 2).  'ab' spells both the keyword KW (literal, priority 1) and an
    identifier (priority 0), and both are viable at the start: KW wins, so 'ab'
    alone is not a sentence although S -> ID would accept it."""
    g = ("start S\ntoken KW \"ab\"\ntoken ID /[a-z]+/\ntoken WS / +/ ignore\n"
         "S : KW ID | ID ;\n")
    o = oracle_mod.Oracle(g)
    assert not o.member(b"ab") and o.member(b"ab cd") and o.member(b"cd")
    assert o.viable(b"ab") and o.viable(b"ab ")
    # an explicit priority on the identifier flips the decision
    g2 = g.replace("token ID /[a-z]+/", "token ID /[a-z]+/ prio 2")
    o2 = oracle_mod.Oracle(g2)
    assert o2.member(b"ab") and not o2.viable(b"ab cd")


def test_equal_priority_ties_go_to_lower_id(oracle_mod):
    """Two terminals with one regex and equal priority: the lower terminal id
    (declaration order) wins the tie."""
    g = ("start S\ntoken A1 /[a-z]+/\ntoken A2 /[a-z]+/\ntoken BANG \"!\"\n"
         "S : A1 BANG | A2 ;\n")
    o = oracle_mod.Oracle(g)
    assert not o.member(b"ab") and o.member(b"ab!")
    g2 = g.replace("S : A1 BANG | A2 ;", "S : A2 BANG | A1 ;")
    o2 = oracle_mod.Oracle(g2)
    assert o2.member(b"ab") and not o2.viable(b"ab!")


def test_consecutive_nullables(oracle_mod):
    """L(S -> A A x, A -> eps | y) = {x, yx, yyx} (up to ignored spaces): two
    nullable nonterminals in a row at one position."""
    g = ("start S\ntoken X \"x\"\ntoken Y \"y\"\ntoken WS / +/ ignore\n"
         "S : A A X ;\nA : %empty | Y ;\n")
    o = oracle_mod.Oracle(g)
    for s, m in [(b"x", 1), (b"yx", 1), (b"yyx", 1), (b"y y x", 1), (b"yyyx", 0), (b"", 0),
                 (b"y", 0), (b"xy", 0)]:
        assert o.member(s) == bool(m), s
    assert o.viable(b"yy") and not o.viable(b"yyy") and not o.viable(b"xx")


def test_nullable_predicted_late(oracle_mod):
    """L(S -> A B, B -> A z, A -> eps | y) = {z, yz, yyz}: the second nullable A
    is predicted only after the first one's empty completion was processed."""
    g = ("start S\ntoken Y \"y\"\ntoken Z \"z\"\n"
         "S : A B ;\nB : A Z ;\nA : %empty | Y ;\n")
    o = oracle_mod.Oracle(g)
    for s, m in [(b"z", 1), (b"yz", 1), (b"yyz", 1), (b"yyyz", 0), (b"y", 0), (b"zz", 0)]:
        assert o.member(s) == bool(m), s


# --------------------------------------------------------------------------
# A third, plain check on random grammars whose lexing is context-free (no
# keywords, no lexicon categories: every lexeme belongs to one terminal):
# maximal munch written out for the generator's token shapes, membership by
# a CYK-style table over the token string, viability by the same table and a
# least fixed point for "this suffix is a prefix of what A derives".  It
# decides Prefix(L) exactly (no completion-length bound), so the oracle's
# viability, membership and mask (Definitions 2 and 4) are compared on every
# string up to 4 bytes over a reduced alphabet.

class _CfgBrute:
    def __init__(self, rg):
        self.prods = rg.prods
        self.start = rg.nts[0]
        self.lit = {v: k for k, v in rg.literal.items()}  # one-byte punctuators
        self.has_num = "NUM" in rg.regex
        self.has_id = "ID" in rg.regex

    def lex(self, w):
        """(emitted terminals, pending lexeme, pending terminal or None, ok):
        a lexeme is emitted when the next byte cannot extend it; the last one
        is pending.  Blank runs are the ignored terminal (pending terminal
        'WS')."""
        s = w.decode("latin-1")
        out, i, n = [], 0, len(s)
        lexemes = []
        while i < n:
            c = s[i]
            if c == " ":
                j = i
                while j < n and s[j] == " ":
                    j += 1
                lexemes.append((s[i:j], "WS"))
            elif c.isdigit():
                j = i
                while j < n and s[j].isdigit():
                    j += 1
                if not self.has_num:
                    return None
                lexemes.append((s[i:j], "NUM"))
            elif "a" <= c <= "z":
                j = i
                while j < n and ("a" <= s[j] <= "z" or s[j].isdigit()):
                    j += 1
                if not self.has_id:
                    return None
                lexemes.append((s[i:j], "ID"))
            elif c in self.lit:
                j = i + 1
                lexemes.append((c, self.lit[c]))
            else:
                return None
            i = j
        if not lexemes:
            return out, None
        for text, t in lexemes[:-1]:
            if t != "WS":
                out.append(t)
        return out, lexemes[-1][1]

    def _tables(self, toks):
        n = len(toks)
        D = {}  # (A, i, j) -> A derives toks[i:j]

        def seq(alt, i, j):
            cur = {i}
            for X in alt:
                nxt = set()
                for p in cur:
                    if X in self.prods:
                        nxt.update(q for q in range(p, j + 1) if D.get((X, p, q)))
                    elif p < j and toks[p] == X:
                        nxt.add(p + 1)
                cur = nxt
                if not cur:
                    return False
            return j in cur

        for L in range(n + 1):
            for i in range(n - L + 1):
                j = i + L
                changed = True
                while changed:
                    changed = False
                    for A, alts in self.prods.items():
                        if not D.get((A, i, j)) and any(seq(alt, i, j) for alt in alts):
                            D[(A, i, j)] = True
                            changed = True
        # P[(A, i)]: toks[i:n] is a prefix of something A derives
        P = {(A, n): True for A in self.prods}
        changed = True
        while changed:
            changed = False
            for i in range(n - 1, -1, -1):
                for A, alts in self.prods.items():
                    if P.get((A, i)):
                        continue
                    ok = False
                    for alt in alts:
                        cur = {i}
                        for X in alt:
                            for p in cur:  # X takes the rest, or part of it
                                if X in self.prods:
                                    if p < n and P.get((X, p)):
                                        ok = True
                                elif p == n - 1 and toks[p] == X:
                                    ok = True
                            if ok:
                                break
                            nxt = set()
                            for p in cur:
                                if X in self.prods:
                                    nxt.update(q for q in range(p, n + 1) if D.get((X, p, q)))
                                elif p < n and toks[p] == X:
                                    nxt.add(p + 1)
                            cur = nxt
                            if n in cur:
                                ok = True
                            if ok or not cur:
                                break
                        if ok:
                            break
                    if ok:
                        P[(A, i)] = True
                        changed = True
        return D, P

    def _prefix(self, toks):
        return bool(self._tables(toks)[1].get((self.start, 0)))

    def _member(self, toks):
        return bool(self._tables(toks)[0].get((self.start, 0, len(toks))))

    def viable(self, w):
        lx = self.lex(w)
        if lx is None:
            return False
        toks, pend = lx
        if pend is None or pend == "WS":
            return self._prefix(toks)
        return self._prefix(toks + [pend])

    def member(self, w):
        lx = self.lex(w)
        if lx is None:
            return False
        toks, pend = lx
        if pend is not None and pend != "WS":
            toks = toks + [pend]
        return self._member(toks)


def test_oracle_matches_cfg_brute_force_on_random_grammars(oracle_mod):
    """Twelve random grammars with context-free lexing (any grammar: Earley
    needs no LALR(1), so ambiguous ones count too): on every string of up to
    4 bytes over a blank, a letter, a digit and the grammar's punctuators the
    oracle's viability equals the CYK check's, and membership (the
    end-of-sequence bit) too; on those up to 3 bytes the whole mask over a
    small vocabulary equals {t : w.t viable}."""
    from workloads.randgram import RandomGrammar
    n_viable = n_checked = 0
    for seed in range(12):
        rg = RandomGrammar(500 + seed, lexicon=False, keywords=False)
        bf = _CfgBrute(rg)
        alpha = [" ", "a", "1"] + list(rg.literal.values())
        vocab = [c.encode() for c in alpha] + [b"a1", b"12", b"1a", b"  ", b"a " + alpha[3].encode(),
                                               (alpha[3] + alpha[-1]).encode(), b""]
        eos = len(vocab) - 1
        o = oracle_mod.Oracle(rg.text(), (), None, vocab, [eos], eos)
        for L in range(5):
            for combo in itertools.product(alpha, repeat=L):
                w = "".join(combo).encode()
                want = bf.viable(w)
                assert o.viable(w) == want, (rg.seed, w, want)
                n_checked += 1
                if not want:
                    continue
                n_viable += 1
                assert o.member(w) == bf.member(w), (rg.seed, w)
                if L <= 3:
                    words, e = o.mask(w, mode=0)
                    bits = np.unpackbits(np.asarray(words, np.uint32).view(np.uint8), bitorder="little")
                    for t, tok in enumerate(vocab[:-1]):
                        assert bool(bits[t]) == bf.viable(w + tok), (rg.seed, w, tok)
                    assert bool(bits[eos]) == bool(e) == bf.member(w), (rg.seed, w)
    assert 0 < n_viable < n_checked


def test_modes_agree_on_random_grammars(oracle_mod):
    """Checkpoint mode (what the GPU parity tests compare against) equals
    from-scratch mode on 16 random grammars with keywords and, in about half
    of them, two lexicon categories sharing the identifier regex: 12 sampled
    prefixes each, the whole mask over the grammar's own 496-token vocabulary."""
    from workloads.randgram import RandomGrammar, random_prefixes, random_vocab
    n_rows = 0
    for seed in range(16):
        rg = RandomGrammar(3000 + seed)
        words = sorted({w for ws in (rg.lexicon or {}).values() for w in ws})
        vocab, specials, eos_id = random_vocab(rg.seed, rg.alphabet(), words=words)
        o = oracle_mod.Oracle(rg.text(), (), rg.lexicon, vocab, specials, eos_id)
        for w in random_prefixes(rg, rg.seed, 12):
            m0, e0 = o.mask(w, mode=0)
            m1, e1 = o.mask(w, mode=1)
            assert np.array_equal(m0, m1) and e0 == e1, (rg.seed, w)
            assert np.asarray(m1).any() or e1, (rg.seed, w)  # a viable prefix has a continuation
            n_rows += 1
    assert n_rows == 16 * 12
