"""Random schema lexicons: table, column and alias names."""

import re
from pathlib import Path

import numpy as np

_LETTERS = np.frombuffer(b"abcdefghijklmnopqrstuvwxyz", dtype=np.uint8)


def keyword_spellings(grammar_path):
    """Lower-cased spellings of the literal tokens declared in a grammar file.

    Identifier names must avoid them so that every lexicon word can win
    contextual resolution whenever its category is allowed.
    """
    out = set()
    for line in Path(grammar_path).read_text().splitlines():
        m = re.match(r'\s*token\s+\w+\s+"([^"]*)"', line)
        if m:
            out.add(m.group(1).lower())
    return out


def random_names(rng, n, lo, hi, banned):
    """n distinct random lowercase names with lengths uniform in [lo, hi]."""
    names = []
    seen = set(banned)
    while len(names) < n:
        k = n - len(names)
        lens = rng.integers(lo, hi + 1, size=2 * k + 8)
        for L in lens:
            s = _LETTERS[rng.integers(0, 26, size=int(L))].tobytes().decode()
            if s in seen:
                continue
            seen.add(s)
            names.append(s)
            if len(names) == n:
                break
    return names


ALIAS_WORDS = [f"t{i}" for i in range(1, 17)] + [f"q{i}" for i in range(1, 9)] + \
    [f"cte{i}" for i in range(1, 9)]


class Schema:
    """Tables (each with its own column list) plus an alias word list."""

    def __init__(self, tables, columns, aliases):
        self.tables = tables            # list[str]
        self.columns = columns          # list[list[str]], per table
        self.aliases = aliases          # list[str]

    def all_columns(self):
        seen = []
        s = set()
        for cols in self.columns:
            for c in cols:
                if c not in s:
                    s.add(c)
                    seen.append(c)
        return seen

    def lexicon(self, with_alias):
        lex = {"TABLE_NAME": list(self.tables), "COLUMN_NAME": self.all_columns()}
        if with_alias:
            lex["ALIAS_NAME"] = list(self.aliases)
        return lex


def make_schema(rng, n_tables, cols_lo, cols_hi, banned, name_lo=4, name_hi=12,
                col_pool=None):
    """Tables and columns with distinct lowercase names.

    Table names and column names are disjoint sets; neither contains a keyword
    spelling.  Column names are drawn from a pool so that tables share some
    columns, as real schemas do.
    """
    tables = random_names(rng, n_tables, name_lo, name_hi, banned)
    ncols = rng.integers(cols_lo, cols_hi + 1, size=n_tables)
    if col_pool is None:
        col_pool = max(int(ncols.sum() * 0.6), int(ncols.max()))
    pool = random_names(rng, col_pool, name_lo, name_hi, set(banned) | set(tables))
    columns = []
    for k in ncols:
        idx = rng.choice(len(pool), size=int(k), replace=False)
        columns.append([pool[i] for i in idx])
    return Schema(tables, columns, list(ALIAS_WORDS))
