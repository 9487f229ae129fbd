"""The five synthetic workloads (seeded), assembled from the generators.

1. expression grammar, V = 1,024, one configuration per call, 64 configurations;
2. SELECT-subset SQL, 8 x 12 schema, V = 32,000, batch 32;
3. full DML SQL with the read-only role projection, 200 x 30 schema,
   V = 151,936, batch 32;
4. the same grammar and projection on 16,000-token sentences with nesting
   depth 1 / 8 / 32 / 128, configurations at positions 1k / 4k / 16k,
   V = 128,256, batch 32 per (position, depth) cell;
5. 256 freshly generated schemas (50..500 tables x 5..60 columns), one row per
   schema, V = 151,936, batch 256, followed by an apply on bf16 logits
   drawn from N(0, 4).

Seeds follow seed = 1000 * workload + k.
"""

import functools
import random
from dataclasses import dataclass, field
from pathlib import Path

import numpy as np

from . import schema as sch
from . import sentences as sen
from . import vocab as voc

GRAMMAR_DIR = Path(__file__).resolve().parent / "grammars"
READ_ONLY_ROLE = ["insert", "update", "delete"]


def grammar_text(name):
    return (GRAMMAR_DIR / f"{name}.grid").read_text()


@dataclass
class Workload:
    name: str
    grammar: str                  # grammar file stem
    drop: list                    # production labels removed by the role projection
    vocab: list                   # list[bytes], index = token id
    specials: list                # special token ids (empty spelling)
    eos_id: int                   # -1 when the vocabulary has no end-of-sequence id
    lexicons: list                # per lexicon slot: {category terminal: [words]}
    prefixes: list                # list[bytes]: the output so far, one per row
    slots: list                   # per row: lexicon slot
    batch: int                    # rows per mask call
    meta: dict = field(default_factory=dict)

    @property
    def V(self):
        return len(self.vocab)

    @property
    def W(self):
        return (self.V + 31) // 32

    def vocab_arrays(self):
        """(bytes uint8[], offsets uint64[V+1]) for the C interfaces."""
        offs = np.zeros(self.V + 1, dtype=np.uint64)
        offs[1:] = np.cumsum([len(t) for t in self.vocab], dtype=np.uint64)
        data = np.frombuffer(b"".join(self.vocab), dtype=np.uint8).copy()
        return data, offs

    def batches(self):
        """Row index lists, one per mask call."""
        n = len(self.prefixes)
        return [list(range(i, min(i + self.batch, n))) for i in range(0, n, self.batch)]


def _truncate(r, text):
    b = text.encode("utf-8")
    return b[: r.randint(0, len(b))]


@functools.lru_cache(maxsize=None)
def _schema3():
    rng = np.random.default_rng(3002)
    banned = sch.keyword_spellings(GRAMMAR_DIR / "sql_dml.grid")
    return sch.make_schema(rng, 200, 30, 30, banned)


@functools.lru_cache(maxsize=None)
def _vocab3():
    kws = sorted(sch.keyword_spellings(GRAMMAR_DIR / "sql_dml.grid"))
    s = _schema3()
    idw = list(s.tables) + s.all_columns()[:2000]
    return voc.geometric_vocab(3000, kws, idw, 151936)


@functools.lru_cache(maxsize=None)
def _vocab4():
    kws = sorted(sch.keyword_spellings(GRAMMAR_DIR / "sql_dml.grid"))
    s = _schema3()
    idw = list(s.tables) + s.all_columns()[:2000]
    return voc.geometric_vocab(4000, kws, idw, 128256)


_TRIES = {}


def _vocab_trie(vocab):
    """Byte trie of a vocabulary's spellings (built once per vocabulary list)."""
    key = id(vocab)
    hit = _TRIES.get(key)
    if hit is not None and hit[0] is vocab:
        return hit[1]
    root = {}
    for tid, sp in enumerate(vocab):
        if not sp:
            continue
        node = root
        for b in sp:
            node = node.setdefault(b, {})
        node[-1] = tid
    _TRIES[key] = (vocab, root)
    return root


def _greedy_tokenize(vocab, text_bytes, max_tokens):
    """Greedy longest-match tokenization; returns byte offsets of token ends."""
    root = _vocab_trie(vocab)
    ends = []
    i = 0
    n = len(text_bytes)
    while i < n and len(ends) < max_tokens:
        node = root
        j = i
        best = -1
        while j < n:
            node = node.get(text_bytes[j])
            if node is None:
                break
            j += 1
            if -1 in node:
                best = j
        assert best > i
        ends.append(best)
        i = best
    return ends


@functools.lru_cache(maxsize=None)
def _long_rows(per_cell):
    """Prefixes and (position, depth, tokens) cells of the 16,000-token workload."""
    s = _schema3()
    vocab, _, _ = _vocab4()
    positions = [1000, 4000, 16000]
    depths = [1, 8, 32, 128]
    prefixes, cells = [], []
    for d in depths:
        r = random.Random(4001 + d)
        g = sen.DmlQueryGen(r, s)
        for j in range(per_cell):
            text = g.long_sentence(d, 100_000).encode("utf-8")
            ends = _greedy_tokenize(vocab, text, max(positions) + 8)
            chain_end = len(text) - 2 * d - 8
            for p in positions:
                n_tok = p - (j % 4)
                cut = ends[n_tok - 1]
                assert cut < chain_end, "sentence too short for the position"
                prefixes.append(text[:cut])
                cells.append((p, d, n_tok))
    # order rows so each batch of per_cell rows is one (position, depth) cell
    order = sorted(range(len(prefixes)), key=lambda i: (cells[i][1], cells[i][0]))
    return tuple(prefixes[i] for i in order), tuple(cells[i] for i in order)


@functools.lru_cache(maxsize=None)
def _long_rows_isolated(per_cell):
    """Prefixes and (position, depth, tokens) cells of the position-isolated
    variant of the 16,000-token workload: per nesting depth one sentence made
    of a header (the nesting) and a fixed block of predicates repeated until
    the text holds more than 16,000 tokens, with no random whitespace, so the
    greedy tokenization is periodic in the repeated part.  The configurations
    at n = 1k / 4k / 16k tokens end at the same offsets inside a block (token
    boundaries that recur in every block), so their local context -- scan
    state, pending bytes and the stack above the chain -- is the same at the
    three positions and only the position differs."""
    s = _schema3()
    vocab, _, _ = _vocab4()
    positions = [1000, 4000, 16000]
    depths = [1, 8, 32, 128]
    prefixes, cells = [], []
    for d in depths:
        r = random.Random(4501 + d)
        g = sen.DmlQueryGen(r, s)
        head, unit = g.periodic_sentence(d)
        head_b, unit_b = head.encode("utf-8"), unit.encode("utf-8")
        reps = 16000 // max(1, len(unit_b) // 8) + 64
        text = head_b + unit_b * reps
        ends = _greedy_tokenize(vocab, text, max(positions) + 4 * len(unit_b))
        ulen, hlen = len(unit_b), len(head_b)

        def unit_of(e):
            return (e - hlen) // ulen, (e - hlen) % ulen

        by_unit = {}
        for i, e in enumerate(ends):
            if e > hlen:
                k, off = unit_of(e)
                by_unit.setdefault(k, {})[off] = i + 1  # tokens up to and including this one
        units = {}
        for p in positions:
            k = unit_of(ends[p - 1])[0] + 1
            units[p] = k
        common = sorted(set.intersection(*(set(by_unit[units[p]]) for p in positions)))
        assert len(common) >= 4, "no recurring token boundaries"
        offs = [common[(j * len(common)) // per_cell % len(common)] for j in range(per_cell)]
        for p in positions:
            k = units[p]
            for off in offs:
                prefixes.append(text[:hlen + k * ulen + off])
                cells.append((p, d, by_unit[k][off]))
    return tuple(prefixes), tuple(cells)


def make_workload(k, n_batches=1, rows=None):
    """Build workload k (1..5; 6 is the position-isolated variant of 4).  n_batches > 1 adds distinct batches of the same
    shape (workloads 2, 3); rows limits the number of rows (tests)."""
    if k == 1:
        vocab = voc.config1_vocab(1000)
        r = random.Random(1001)
        n = 64 if rows is None else rows
        prefixes = [_truncate(r, sen.gen_expr(r)) for _ in range(n)]
        return Workload("expr", "expr", [], vocab, [], -1, [{}], prefixes,
                        [0] * n, 1)
    if k == 2:
        rng = np.random.default_rng(2002)
        banned = sch.keyword_spellings(GRAMMAR_DIR / "sql_select.grid")
        s = sch.make_schema(rng, 8, 12, 12, banned)
        kws = sorted(banned)
        vocab, specials, eos = voc.config2_vocab(2000, kws, list(s.tables) + s.all_columns())
        r = random.Random(2001)
        g = sen.SelectSubsetGen(r, s)
        n = 32 * n_batches if rows is None else rows
        prefixes = [_truncate(r, g.sentence()) for _ in range(n)]
        return Workload("sql_select", "sql_select", [], vocab, specials, eos,
                        [s.lexicon(with_alias=False)], prefixes, [0] * n, 32,
                        meta={"schema": s})
    if k == 3:
        s = _schema3()
        vocab, specials, eos = _vocab3()
        r = random.Random(3001)
        g = sen.DmlQueryGen(r, s)
        n = 32 * n_batches if rows is None else rows
        prefixes = [_truncate(r, g.sentence()) for _ in range(n)]
        return Workload("sql_dml_ro", "sql_dml", list(READ_ONLY_ROLE), vocab, specials, eos,
                        [s.lexicon(with_alias=True)], prefixes, [0] * n, 32,
                        meta={"schema": s})
    if k == 4:
        s = _schema3()
        vocab, specials, eos = _vocab4()
        per_cell = 32 if rows is None else rows
        prefixes, cells = _long_rows(per_cell)
        return Workload("sql_dml_long", "sql_dml", list(READ_ONLY_ROLE), vocab, specials, eos,
                        [s.lexicon(with_alias=True)], list(prefixes), [0] * len(prefixes), per_cell,
                        meta={"cells": list(cells), "schema": s})
    if k == 5:
        vocab, specials, eos = _vocab3()
        banned = sch.keyword_spellings(GRAMMAR_DIR / "sql_dml.grid")
        n = 256 if rows is None else rows
        lexicons, prefixes, schemas = [], [], []
        for i in range(n):
            rng = np.random.default_rng(5000 + 7 * i)
            nt = int(rng.integers(50, 501))
            s = sch.make_schema(rng, nt, 5, 60, banned)
            r = random.Random(5001 + 7 * i)
            g = sen.DmlQueryGen(r, s)
            prefixes.append(_truncate(r, g.sentence()))
            lexicons.append(s.lexicon(with_alias=True))
            schemas.append(s)
        return Workload("sql_dml_cold_schema", "sql_dml", list(READ_ONLY_ROLE), vocab,
                        specials, eos, lexicons, prefixes, list(range(n)), n,
                        meta={"logits_seed": 5999, "logits_std": 2.0})
    if k == 6:
        s = _schema3()
        vocab, specials, eos = _vocab4()
        per_cell = 32 if rows is None else rows
        prefixes, cells = _long_rows_isolated(per_cell)
        return Workload("sql_dml_long_isolated", "sql_dml", list(READ_ONLY_ROLE), vocab, specials, eos,
                        [s.lexicon(with_alias=True)], list(prefixes), [0] * len(prefixes), per_cell,
                        meta={"cells": list(cells), "schema": s})
    raise ValueError(f"no workload {k}")
