"""Synthetic byte-level token vocabularies.

A vocabulary is a list of byte strings indexed by token id.  Special tokens
(end-of-sequence and the like) have the empty spelling.
"""

import numpy as np

SQL_PUNCT = [",", ".", ";", "(", ")", "*", "+", "-", "/", "=", "<", ">", "<=", ">=", "<>",
             "!=", "'", "%", "||", "),", ");", "(*)", " =", " (", ", ", " *", "')", "',",
             " '", "();", "))", "((", "')", " >", " <", "--", "\n", "  ", "   ", "\n  "]


def _case_variants(word):
    return [word.lower(), word.upper(), word.capitalize()]


def config1_vocab(seed):
    """256 single bytes plus 768 strings of length 2..8 over [0-9a-z+*() ]."""
    rng = np.random.default_rng(seed)
    alphabet = np.frombuffer(b"0123456789abcdefghijklmnopqrstuvwxyz+*() ", dtype=np.uint8)
    vocab = [bytes([b]) for b in range(256)]
    for _ in range(768):
        L = int(rng.integers(2, 9))
        vocab.append(alphabet[rng.integers(0, len(alphabet), size=L)].tobytes())
    return vocab


def _sqlish_pool(keywords, ident_words, rng, n_ident_frag):
    pool = set()
    for kw in keywords:
        for v in _case_variants(kw):
            for i in range(len(v)):
                for j in range(i + 1, len(v) + 1):
                    pool.add(v[i:j].encode())
                    if i == 0:
                        pool.add((" " + v[:j]).encode())
    words = list(ident_words)
    for _ in range(n_ident_frag):
        w = words[int(rng.integers(0, len(words)))]
        i = int(rng.integers(0, len(w)))
        j = int(rng.integers(i + 1, len(w) + 1))
        frag = w[i:j]
        pool.add(frag.encode())
        if rng.random() < 0.5:
            pool.add((" " + frag).encode())
    for L in range(1, 7):
        for _ in range(60 * L):
            pool.add("".join(str(int(d)) for d in rng.integers(0, 10, size=L)).encode())
    for p in SQL_PUNCT:
        pool.add(p.encode())
    return pool


def config2_vocab(seed, keywords, ident_words, V=32000):
    """BPE-like vocabulary for the SELECT-subset workload.

    256 single bytes; keyword substrings with and without a leading space in
    three letter cases; identifier fragments of the schema names; digit runs;
    punctuation clusters; 20% random printable-ASCII strings of 2..12 chars.
    Ids V-2 (a begin marker) and V-1 (end of sequence) are special.
    """
    rng = np.random.default_rng(seed)
    n_special = 2
    n_random = V // 5
    n_sqlish = V - 256 - n_random - n_special
    pool = _sqlish_pool(keywords, ident_words, rng, 4 * n_sqlish)
    pool = sorted(p for p in pool if len(p) >= 2)
    pick = rng.choice(len(pool), size=min(n_sqlish, len(pool)), replace=False)
    sqlish = [pool[i] for i in pick]
    seen = set(sqlish) | {bytes([b]) for b in range(256)}
    printable = np.arange(32, 127, dtype=np.uint8)
    rand = []
    while len(rand) < n_random + (n_sqlish - len(sqlish)):
        L = int(rng.integers(2, 13))
        s = printable[rng.integers(0, len(printable), size=L)].tobytes()
        if s not in seen:
            seen.add(s)
            rand.append(s)
    body = sqlish + rand
    order = rng.permutation(len(body))
    vocab = [bytes([b]) for b in range(256)] + [body[i] for i in order]
    vocab += [b"", b""]
    assert len(vocab) == V
    return vocab, [V - 2, V - 1], V - 1


def _utf8_chunk(rng):
    ranges = [(0xA0, 0x24F), (0x370, 0x3FF), (0x400, 0x4FF), (0x4E00, 0x9FFF),
              (0x3040, 0x30FF), (0x1F300, 0x1F64F)]
    lo, hi = ranges[int(rng.integers(0, len(ranges)))]
    return chr(int(rng.integers(lo, hi + 1))).encode("utf-8")


def geometric_vocab(seed, keywords, ident_words, V, n_alias=None):
    """Byte-level vocabulary whose lengths are geometric with mean 4, max 32.

    256 single bytes at ids 0..255; the other spellings have length
    1 + Geometric(1/3) (resampled above 32), 40% SQL-ish fragments built from
    keyword pieces, identifier fragments, digits, punctuation and spaces, 60%
    random bytes of which half are valid multi-byte UTF-8 text.  A small number
    of ids repeat an earlier spelling (alias classes).  Id V-1 is the special
    end-of-sequence token.
    """
    rng = np.random.default_rng(seed)
    if n_alias is None:
        n_alias = V // 500
    n_body = V - 256 - 1 - n_alias
    kw_pieces = []
    for kw in keywords:
        for v in _case_variants(kw):
            kw_pieces.append(v.encode())
            kw_pieces.append((" " + v).encode())
    idw = [w.encode() for w in ident_words]
    punct = [p.encode() for p in SQL_PUNCT]
    seen = {bytes([b]) for b in range(256)}
    body = []

    def draw_len():
        while True:
            L = 1 + int(rng.geometric(1.0 / 3.0))
            if L <= 32:
                return L

    while len(body) < n_body:
        L = draw_len()
        if rng.random() < 0.4:
            parts = []
            n = 0
            while n < L + 1:
                k = rng.random()
                if k < 0.35:
                    p = kw_pieces[int(rng.integers(0, len(kw_pieces)))]
                elif k < 0.65:
                    w = idw[int(rng.integers(0, len(idw)))]
                    i = int(rng.integers(0, len(w)))
                    p = w[i:]
                    if rng.random() < 0.4:
                        p = b" " + p
                elif k < 0.75:
                    p = str(int(rng.integers(0, 10 ** int(rng.integers(1, 6))))).encode()
                elif k < 0.95:
                    p = punct[int(rng.integers(0, len(punct)))]
                else:
                    p = b" "
                parts.append(p)
                n += len(p)
            s = b"".join(parts)
            start = int(rng.integers(0, max(1, min(len(s) - L, 3) + 1)))
            s = s[start:start + L]
        elif rng.random() < 0.5:
            s = rng.integers(0, 256, size=L, dtype=np.uint8).tobytes()
        else:
            chunks = []
            n = 0
            while n < L:
                c = _utf8_chunk(rng) if rng.random() < 0.7 else bytes(
                    [int(rng.integers(32, 127))])
                chunks.append(c)
                n += len(c)
            s = b"".join(chunks)[:L]
        if len(s) != L or s in seen:
            continue
        seen.add(s)
        body.append(s)
    alias_src = rng.integers(0, len(body), size=n_alias)
    body += [body[int(i)] for i in alias_src]
    order = rng.permutation(len(body))
    vocab = [bytes([b]) for b in range(256)] + [body[i] for i in order] + [b""]
    assert len(vocab) == V
    return vocab, [V - 1], V - 1
