"""Seeded random grammars in the .grid format, sentences sampled from them and
a small vocabulary over their bytes.

Inputs for tests that compare the GPU path with the oracle (and the kernels'
rewritten LR tables with the plain LALR ones) beyond the five fixed grammars:
chains of one-symbol productions, empty productions, left and right
recursion, bracketed nesting and keywords that a regex terminal also
matches.  Many random grammars are not LALR(1); a caller keeps the seeds whose
grammar compiles.  Nothing here computes any part of a mask.
"""

import random

PUNCT = ["(", ")", "+", ",", ";", "[", "]", "-", "=", ".", ":", "*"]
KEYWORDS = ["if", "do", "end", "let", "or"]
BRACKETS = [("(", ")"), ("[", "]")]


class RandomGrammar:
    """A random grammar: terminals (punctuators, keywords, NUM, ID, ignored
    blanks) and nonterminals N0 (the start) .. N{n-1}, each with one to four
    alternatives.  Every nonterminal has an alternative that refers only to
    terminals and higher-numbered nonterminals, so every one derives a
    terminal string, and N0 reaches every other one.  With lexicon=True (or
    at random when it is None) ID gives way to two lexicon categories CA and
    CB that share its regex, with word lists over a few letters (many words
    prefixes of others) in self.lexicon.  keywords=False and lexicon=False
    give a grammar whose lexemes each belong to one terminal only."""

    def __init__(self, seed, n_nt=None, lexicon=None, keywords=True):
        r = random.Random(seed)
        self.seed = seed
        n = n_nt if n_nt is not None else r.randint(3, 7)
        punct = r.sample(PUNCT, r.randint(3, 7))
        kws = r.sample(KEYWORDS, r.randint(0, 2))
        if not keywords:
            kws = []
        self.literal = {}  # terminal name -> its text
        for i, p in enumerate(punct):
            self.literal[f"P{i}"] = p
        for kw in kws:
            self.literal[f"K{kw.upper()}"] = kw
        self.regex = {"NUM": "[0-9]+", "ID": "[a-z][a-z0-9]*"}
        if r.random() < 0.3:
            del self.regex["NUM"]
        self.lexicon = None
        if lexicon if lexicon is not None else r.random() < 0.5:
            del self.regex["ID"]
            self.regex["CA"] = self.regex["CB"] = "[a-z]+"
            kw = set(self.literal.values())
            self.lexicon = {}
            for cat in ("CA", "CB"):
                words = set()
                while len(words) < r.randint(3, 9):
                    w = "".join(r.choice("abcdef") for _ in range(r.randint(1, 5)))
                    if w not in kw and all(w not in ws for ws in self.lexicon.values()):
                        words.add(w)  # the two lists are disjoint: a word names its category
                self.lexicon[cat] = sorted(words)
        terms = list(self.literal) + list(self.regex)
        # brackets used by nesting alternatives when both halves were drawn
        by_text = {v: k for k, v in self.literal.items()}
        pairs = [(by_text[a], by_text[b]) for a, b in BRACKETS if a in by_text and b in by_text]
        self.nts = [f"N{i}" for i in range(n)]
        self.prods = {}
        for i, a in enumerate(self.nts):
            below = self.nts[i + 1:]
            alts = []
            # the terminating alternative
            if below and r.random() < 0.5:
                alts.append([r.choice(below)])  # a one-symbol production
            elif r.random() < 0.15 and i > 0:
                alts.append([])  # an empty production
            else:
                alts.append([r.choice(terms) for _ in range(r.randint(1, 2))] +
                            ([r.choice(below)] if below and r.random() < 0.5 else []))
            for _ in range(r.randint(0, 3)):
                kind = r.random()
                if kind < 0.2 and pairs:  # bracketed nesting back to the start or to itself
                    lb, rb = r.choice(pairs)
                    alts.append([lb, r.choice([self.nts[0], a]), rb])
                elif kind < 0.45:  # left or right recursion through a terminal
                    t = r.choice(terms)
                    alts.append([a, t] + ([r.choice(below)] if below else [r.choice(terms)]) if r.random() < 0.5
                                else ([r.choice(below)] if below else [r.choice(terms)]) + [t, a])
                elif kind < 0.6 and below:
                    alts.append([r.choice(below)])
                elif kind < 0.7 and i > 0:
                    alts.append([])
                else:
                    body = [r.choice(terms + below) for _ in range(r.randint(1, 3))]
                    alts.append(body)
            # at most one empty alternative, no duplicates
            seen, uniq = set(), []
            for alt in alts:
                key = tuple(alt)
                if key not in seen:
                    seen.add(key)
                    uniq.append(alt)
            self.prods[a] = uniq
        # every nonterminal reachable from N0: N{i} for i > 0 not yet used
        # becomes an extra alternative of some lower one
        used = {self.nts[0]}
        for a in self.nts:
            for alt in self.prods[a]:
                used.update(s for s in alt if s in self.prods)
        for i, a in enumerate(self.nts[1:], start=1):
            if a not in used:
                host = self.nts[r.randrange(i)]
                self.prods[host].append([r.choice(terms), a])
                used.add(a)
        self._heights_of = {}

    def label(self, a, k):
        """The label of nonterminal a's k-th alternative (role projections
        drop alternatives by label)."""
        return f"{a}_{k}"

    def labels(self):
        return [self.label(a, k) for a in self.nts for k in range(len(self.prods[a]))]

    def _alts(self, a, drop):
        return [alt for k, alt in enumerate(self.prods[a]) if self.label(a, k) not in drop]

    def _heights(self, drop=()):
        """Least derivation depth of each nonterminal once the alternatives
        labelled in drop are gone (None: it derives no terminal string)."""
        key = tuple(sorted(drop))
        if key in self._heights_of:
            return self._heights_of[key]
        h = {a: None for a in self.nts}
        changed = True
        while changed:
            changed = False
            for a in self.nts:
                for alt in self._alts(a, drop):
                    sub = [h[s] for s in alt if s in h]
                    if any(x is None for x in sub):
                        continue
                    v = 1 + max(sub, default=0)
                    if h[a] is None or v < h[a]:
                        h[a] = v
                        changed = True
        self._heights_of[key] = h
        return h

    def random_drop(self, r, n):
        """n labels to drop, at random."""
        return r.sample(self.labels(), min(n, len(self.labels())))

    def text(self):
        out = [f"# random grammar, seed {self.seed}", "start N0", ""]
        for name, lit in self.literal.items():
            out.append(f'token {name} "{lit}"')
        for name, rx in self.regex.items():
            out.append(f"token {name} /{rx}/" + (" category" if name in ("CA", "CB") else ""))
        out.append("token WS /[ ]+/ ignore")
        out.append("")
        for a in self.nts:
            alts = [(" ".join(alt) if alt else "%empty") + f" @{self.label(a, k)}"
                    for k, alt in enumerate(self.prods[a])]
            out.append(f"{a} : {' | '.join(alts)} ;")
        return "\n".join(out) + "\n"

    def _lexeme(self, r, t):
        if t in self.literal:
            return self.literal[t]
        if t == "NUM":
            return str(r.randint(0, 999))
        if t in ("CA", "CB"):
            return r.choice(self.lexicon[t])
        while True:  # an identifier that is no keyword
            w = "".join(r.choice("abcdefghijklmnopqrstuvwxyz") for _ in range(r.randint(1, 4)))
            if w not in self.literal.values():
                return w

    def sentence(self, r, max_depth=7, max_len=60, drop=()):
        """A random member of the language (of its projection without the
        alternatives labelled in drop): a derivation that takes the
        shallowest alternative below the depth limit, lexemes joined by one
        blank (so maximal munch splits them where they were joined)."""
        out = []
        h = self._heights(drop)
        assert h[self.nts[0]] is not None, "the projection leaves an empty language"

        def height(alt):
            sub = [h[s] for s in alt if s in h]
            return None if any(x is None for x in sub) else 1 + max(sub, default=0)

        def expand(a, d):
            alts = [alt for alt in self._alts(a, drop) if height(alt) is not None]
            if d >= max_depth or len(out) > max_len:
                best = min(height(alt) for alt in alts)
                alts = [alt for alt in alts if height(alt) == best]
            for s in r.choice(alts):
                if s in self.prods:
                    expand(s, d + 1)
                else:
                    out.append(self._lexeme(r, s))

        expand(self.nts[0], 0)
        return " ".join(out).encode()

    def alphabet(self):
        """The bytes the grammar's lexemes and blanks use."""
        chars = set(" ") | set("".join(self.literal.values()))
        if "NUM" in self.regex:
            chars |= set("0123456789")
        chars |= set("abcdefghijklmnopqrstuvwxyz0123456789")
        return sorted(chars)


def random_vocab(seed, alphabet, n_multi=400, eos=True, words=()):
    """Every printable ASCII byte as a token, then the given words, each also
    with a leading blank, then distinct strings of 2..6 bytes over the
    grammar's alphabet (a few with a leading blank) up to n_multi beyond the
    bytes, and an end-of-sequence special with an empty spelling last."""
    r = random.Random(seed)
    vocab = [bytes([b]) for b in range(0x20, 0x7F)]
    seen = set(vocab)
    for w in words:
        for t in (w.encode(), (" " + w).encode()):
            if t not in seen and len(vocab) < 95 + n_multi:
                seen.add(t)
                vocab.append(t)
    while len(vocab) < 95 + n_multi:
        s = "".join(r.choice(alphabet) for _ in range(r.randint(2, 6)))
        if r.random() < 0.2:
            s = " " + s[1:]
        t = s.encode()
        if t not in seen:
            seen.add(t)
            vocab.append(t)
    specials, eos_id = [], -1
    if eos:
        eos_id = len(vocab)
        vocab.append(b"")
        specials = [eos_id]
    return vocab, specials, eos_id


def random_prefixes(g, seed, n, drop=()):
    """n viable prefixes: random sentences cut at random byte offsets, with
    the empty prefix and whole sentences among them."""
    r = random.Random(seed)
    out = [b""]
    while len(out) < n:
        s = g.sentence(r, drop=drop)
        cut = len(s) if r.random() < 0.15 else r.randint(0, len(s))
        out.append(s[:cut])
    return out
