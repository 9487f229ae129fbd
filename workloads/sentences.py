"""Random sentences of the workload languages.

Each generator writes lexemes separated by whitespace following the grammar
shapes by hand; the tests confirm with the oracle that the sentences are
members of the language.  Keywords get random letter case; identifiers come
from the schema so every identifier lexeme is in its lexicon.
"""

import random


# ---------------------------------------------------------------- expressions
def gen_expr(r: random.Random, max_depth=6):
    """A random expression of the E/T/F grammar with paren nesting <= max_depth."""

    def ws():
        return " " * r.choice([0, 0, 0, 1, 1, 2])

    def num():
        return "".join(r.choice("0123456789") for _ in range(r.randint(1, 4)))

    def ident():
        first = r.choice("abcdefghijklmnopqrstuvwxyz")
        rest = "".join(r.choice("abcdefghijklmnopqrstuvwxyz0123456789")
                       for _ in range(r.randint(0, 5)))
        return first + rest

    def F(d):
        k = r.random()
        if d < max_depth and k < 0.3:
            return "(" + ws() + E(d + 1) + ws() + ")"
        return num() if k < 0.65 else ident()

    def T(d):
        parts = [F(d)]
        while r.random() < 0.35:
            parts.append(F(d))
        return (ws() + "*" + ws()).join(parts)

    def E(d):
        parts = [T(d)]
        while r.random() < 0.4:
            parts.append(T(d))
        # a space is needed between adjacent operands only; operators separate here
        return (ws() + "+" + ws()).join(parts)

    return E(0)


# ------------------------------------------------------------------------ SQL
class _SqlWriter:
    """Collects lexemes and joins them with random (safe) whitespace."""

    TIGHT = {",", "(", ")", ";", "."}

    def __init__(self, r):
        self.r = r
        self.out = []

    def kw(self, word):
        c = self.r.random()
        if c < 0.55:
            w = word.lower()
        elif c < 0.85:
            w = word.upper()
        else:
            w = word.capitalize()
        self.out.append(w)

    def lit(self, s):
        self.out.append(s)

    def text(self, comments=False):
        r = self.r
        parts = []
        prev = None
        for lx in self.out:
            if prev is not None:
                if (lx in self.TIGHT or prev in self.TIGHT) and r.random() < 0.5:
                    sep = ""
                else:
                    c = r.random()
                    sep = " " if c < 0.85 else ("\n" if c < 0.93 else "  ")
                    if comments and r.random() < 0.01:
                        sep = " -- note " + str(r.randint(0, 99)) + "\n"
                parts.append(sep)
            parts.append(lx)
            prev = lx
        return "".join(parts)


def _string_lit(r):
    alphabet = "abcdefghijklmnopqrstuvwxyz ABCDEFGHIJ0123456789_-.,:%"
    body = "".join(r.choice(alphabet) for _ in range(r.randint(0, 10)))
    if r.random() < 0.15:
        body += r.choice(["é", "ß", "日本", "π", "€"])
    return "'" + body + "'"


class SelectSubsetGen:
    """Sentences of the SELECT-subset grammar."""

    def __init__(self, r, schema, max_bool_depth=2):
        self.r = r
        self.s = schema
        self.maxd = max_bool_depth

    def sentence(self):
        w = _SqlWriter(self.r)
        self.select_stmt(w)
        w.lit(";")
        return w.text()

    def table(self):
        return self.r.randrange(len(self.s.tables))

    def column_ref(self, w, tabs):
        r = self.r
        t = r.choice(tabs)
        c = r.choice(self.s.columns[t])
        if r.random() < 0.3:
            w.lit(self.s.tables[t])
            w.lit(".")
        w.lit(c)

    def value(self, w, tabs, depth=0):
        r = self.r
        self.term(w, tabs, depth)
        while r.random() < 0.2:
            w.lit(r.choice(["+", "-"]))
            self.term(w, tabs, depth)

    def term(self, w, tabs, depth):
        r = self.r
        self.factor(w, tabs, depth)
        while r.random() < 0.15:
            w.lit(r.choice(["*", "/"]))
            self.factor(w, tabs, depth)

    def factor(self, w, tabs, depth):
        r = self.r
        k = r.random()
        if k < 0.55:
            self.column_ref(w, tabs)
        elif k < 0.75:
            w.lit(str(r.randint(0, 99999)))
        elif k < 0.85:
            w.lit(_string_lit(r))
        elif k < 0.9 and depth < 3:
            # "-" is never written flush against a neighbour, so "- -x" stays two lexemes
            w.lit("-")
            self.factor(w, tabs, depth + 1)
        else:
            fn = r.choice(["COUNT", "SUM", "AVG", "MIN", "MAX"])
            w.kw(fn)
            w.lit("(")
            if fn == "COUNT" and r.random() < 0.5:
                w.lit("*")
            else:
                self.value(w, tabs, depth + 1)
            w.lit(")")

    def predicate(self, w, tabs):
        r = self.r
        k = r.random()
        if k < 0.5:
            self.value(w, tabs)
            w.lit(r.choice(["=", "<>", "!=", "<", "<=", ">", ">="]))
            self.value(w, tabs)
        elif k < 0.6:
            self.value(w, tabs)
            w.kw("IS")
            if r.random() < 0.5:
                w.kw("NOT")
            w.kw("NULL")
        elif k < 0.7:
            self.value(w, tabs)
            w.kw("LIKE")
            w.lit(_string_lit(r))
        elif k < 0.8:
            self.value(w, tabs)
            w.kw("BETWEEN")
            self.value(w, tabs)
            w.kw("AND")
            self.value(w, tabs)
        elif k < 0.95:
            self.value(w, tabs)
            if r.random() < 0.3:
                w.kw("NOT")
            w.kw("IN")
            w.lit("(")
            self.value(w, tabs)
            for _ in range(r.randint(0, 3)):
                w.lit(",")
                self.value(w, tabs)
            w.lit(")")
        else:
            w.kw(r.choice(["TRUE", "FALSE"]))

    def bool_expr(self, w, tabs, d=0):
        r = self.r
        self.bool_term(w, tabs, d)
        while r.random() < 0.25:
            w.kw("OR")
            self.bool_term(w, tabs, d)

    def bool_term(self, w, tabs, d):
        r = self.r
        self.bool_factor(w, tabs, d)
        while r.random() < 0.35:
            w.kw("AND")
            self.bool_factor(w, tabs, d)

    def bool_factor(self, w, tabs, d):
        r = self.r
        k = r.random()
        if k < 0.1:
            w.kw("NOT")
            self.bool_factor(w, tabs, d)
        elif k < 0.25 and d < self.maxd:
            w.lit("(")
            self.bool_expr(w, tabs, d + 1)
            w.lit(")")
        else:
            self.predicate(w, tabs)

    def select_stmt(self, w):
        r = self.r
        tabs = [self.table()]
        w.kw("SELECT")
        if r.random() < 0.15:
            w.kw("DISTINCT")
        sel_mark = len(w.out)
        w.kw("FROM")
        w.lit(self.s.tables[tabs[0]])
        from_part = w.out[sel_mark:]
        del w.out[sel_mark:]
        joins = []
        while r.random() < 0.3:
            t = self.table()
            jw = _SqlWriter(r)
            kind = r.random()
            if kind < 0.25:
                jw.kw("INNER")
            elif kind < 0.45:
                jw.kw("LEFT")
            elif kind < 0.55:
                jw.kw("LEFT")
                jw.kw("OUTER")
            jw.kw("JOIN")
            jw.lit(self.s.tables[t])
            jw.kw("ON")
            tabs.append(t)
            self.bool_expr(jw, tabs)
            joins.append(jw.out)
        # select list may reference any joined table
        if r.random() < 0.2:
            w.lit("*")
        else:
            self.value(w, tabs)
            for _ in range(r.randint(0, 3)):
                w.lit(",")
                self.value(w, tabs)
        w.out.extend(from_part)
        for j in joins:
            w.out.extend(j)
        if r.random() < 0.7:
            w.kw("WHERE")
            self.bool_expr(w, tabs)
        if r.random() < 0.2:
            w.kw("GROUP")
            w.kw("BY")
            self.column_ref(w, tabs)
            for _ in range(r.randint(0, 2)):
                w.lit(",")
                self.column_ref(w, tabs)
            if r.random() < 0.4:
                w.kw("HAVING")
                self.bool_expr(w, tabs)
        if r.random() < 0.3:
            w.kw("ORDER")
            w.kw("BY")
            n = r.randint(1, 3)
            for i in range(n):
                if i:
                    w.lit(",")
                self.value(w, tabs)
                c = r.random()
                if c < 0.3:
                    w.kw("ASC")
                elif c < 0.6:
                    w.kw("DESC")
        if r.random() < 0.3:
            w.kw("LIMIT")
            w.lit(str(r.randint(1, 1000)))


class DmlQueryGen:
    """Read-only sentences (queries) of the full DML grammar."""

    def __init__(self, r, schema, max_depth=3):
        self.r = r
        self.s = schema
        self.maxd = max_depth

    def sentence(self, comments=True):
        w = _SqlWriter(self.r)
        self.query_stmt(w, 0)
        w.lit(";")
        return w.text(comments=comments)

    # -- names
    def tname(self):
        return self.r.randrange(len(self.s.tables))

    def alias(self):
        return self.r.choice(self.s.aliases)

    def column_ref(self, w, scope):
        r = self.r
        t, al = r.choice(scope)
        c = r.choice(self.s.columns[t]) if t is not None else \
            r.choice(self.s.columns[r.randrange(len(self.s.tables))])
        k = r.random()
        if al is not None and k < 0.4:
            w.lit(al)
            w.lit(".")
        elif t is not None and k < 0.55:
            w.lit(self.s.tables[t])
            w.lit(".")
        w.lit(c)

    # -- values
    def value(self, w, scope, d):
        r = self.r
        self.term(w, scope, d)
        while r.random() < 0.2:
            w.lit(r.choice(["+", "-", "||"]))
            self.term(w, scope, d)

    def term(self, w, scope, d):
        r = self.r
        self.factor(w, scope, d)
        while r.random() < 0.12:
            w.lit(r.choice(["*", "/", "%"]))
            self.factor(w, scope, d)

    def factor(self, w, scope, d):
        r = self.r
        if r.random() < 0.05 and d < self.maxd + 2:
            w.lit(r.choice(["-", "+"]))
            self.factor(w, scope, d + 1)
            return
        self.primary(w, scope, d)

    def primary(self, w, scope, d):
        r = self.r
        k = r.random()
        if k < 0.5:
            self.column_ref(w, scope)
        elif k < 0.62:
            w.lit(str(r.randint(0, 99999)))
        elif k < 0.67:
            w.lit(f"{r.randint(0, 999)}.{r.randint(0, 99)}")
        elif k < 0.75:
            w.lit(_string_lit(r))
        elif k < 0.77:
            w.kw("NULL")
        elif k < 0.87:
            self.func(w, scope, d)
        elif k < 0.9 and d < self.maxd:
            w.kw("CASE")
            for _ in range(r.randint(1, 2)):
                w.kw("WHEN")
                self.bool_expr(w, scope, d + 1)
                w.kw("THEN")
                self.value(w, scope, d + 1)
            if r.random() < 0.5:
                w.kw("ELSE")
                self.value(w, scope, d + 1)
            w.kw("END")
        elif k < 0.93 and d < self.maxd:
            w.kw("CAST")
            w.lit("(")
            self.value(w, scope, d + 1)
            w.kw("AS")
            w.kw(r.choice(["INTEGER", "TEXT", "REAL", "DATE"]))
            w.lit(")")
        elif k < 0.97 and d < self.maxd:
            w.lit("(")
            self.value(w, scope, d + 1)
            w.lit(")")
        elif d < self.maxd:
            w.lit("(")
            self.query_stmt(w, d + 1)
            w.lit(")")
        else:
            self.column_ref(w, scope)

    def func(self, w, scope, d):
        r = self.r
        k = r.random()
        if k < 0.3:
            w.kw("COUNT")
            w.lit("(")
            c = r.random()
            if c < 0.5:
                w.lit("*")
            else:
                if c < 0.65:
                    w.kw("DISTINCT")
                self.value(w, scope, d + 1)
            w.lit(")")
        elif k < 0.6:
            w.kw(r.choice(["SUM", "AVG", "MIN", "MAX"]))
            w.lit("(")
            if r.random() < 0.1:
                w.kw("DISTINCT")
            self.value(w, scope, d + 1)
            w.lit(")")
        else:
            w.kw(r.choice(["UPPER", "LOWER", "LENGTH", "ABS", "ROUND", "COALESCE"]))
            w.lit("(")
            self.value(w, scope, d + 1)
            for _ in range(r.randint(0, 1)):
                w.lit(",")
                self.value(w, scope, d + 1)
            w.lit(")")

    # -- booleans
    def predicate(self, w, scope, d):
        r = self.r
        k = r.random()
        if k < 0.45:
            self.value(w, scope, d)
            w.lit(r.choice(["=", "<>", "!=", "<", "<=", ">", ">="]))
            self.value(w, scope, d)
        elif k < 0.53:
            self.value(w, scope, d)
            w.kw("IS")
            if r.random() < 0.5:
                w.kw("NOT")
            w.kw("NULL")
        elif k < 0.6:
            self.value(w, scope, d)
            if r.random() < 0.3:
                w.kw("NOT")
            w.kw("LIKE")
            w.lit(_string_lit(r))
        elif k < 0.67:
            self.value(w, scope, d)
            if r.random() < 0.3:
                w.kw("NOT")
            w.kw("BETWEEN")
            self.value(w, scope, d)
            w.kw("AND")
            self.value(w, scope, d)
        elif k < 0.8:
            self.value(w, scope, d)
            if r.random() < 0.3:
                w.kw("NOT")
            w.kw("IN")
            w.lit("(")
            if d < self.maxd and r.random() < 0.4:
                self.query_stmt(w, d + 1)
            else:
                self.value(w, scope, d)
                for _ in range(r.randint(0, 3)):
                    w.lit(",")
                    self.value(w, scope, d)
            w.lit(")")
        elif k < 0.86 and d < self.maxd:
            w.kw("EXISTS")
            w.lit("(")
            self.query_stmt(w, d + 1)
            w.lit(")")
        elif k < 0.9:
            w.kw(r.choice(["TRUE", "FALSE"]))
        else:
            self.value(w, scope, d)
            w.lit("=")
            self.value(w, scope, d)

    def bool_expr(self, w, scope, d):
        r = self.r
        self.bool_term(w, scope, d)
        while r.random() < 0.2:
            w.kw("OR")
            self.bool_term(w, scope, d)

    def bool_term(self, w, scope, d):
        r = self.r
        self.bool_factor(w, scope, d)
        while r.random() < 0.3:
            w.kw("AND")
            self.bool_factor(w, scope, d)

    def bool_factor(self, w, scope, d):
        r = self.r
        k = r.random()
        if k < 0.08:
            w.kw("NOT")
            self.bool_factor(w, scope, d)
        elif k < 0.2 and d < self.maxd:
            w.lit("(")
            self.bool_expr(w, scope, d + 1)
            w.lit(")")
        else:
            self.predicate(w, scope, d)

    # -- queries
    def table_ref(self, w, d, scope):
        r = self.r
        k = r.random()
        if k < 0.1 and d < self.maxd:
            w.lit("(")
            self.query_stmt(w, d + 1)
            w.lit(")")
            al = self.alias()
            if r.random() < 0.5:
                w.kw("AS")
            w.lit(al)
            scope.append((None, al))
            return
        t = self.tname()
        w.lit(self.s.tables[t])
        al = None
        if k < 0.5:
            al = self.alias()
            if r.random() < 0.5:
                w.kw("AS")
            w.lit(al)
        scope.append((t, al))

    def select_core(self, w, d):
        r = self.r
        w.kw("SELECT")
        c = r.random()
        if c < 0.1:
            w.kw("DISTINCT")
        elif c < 0.13:
            w.kw("ALL")
        # build FROM first (scope), then the select list
        fw = _SqlWriter(r)
        scope = []
        has_from = r.random() < 0.95
        if has_from:
            fw.kw("FROM")
            self.table_ref(fw, d, scope)
            while r.random() < 0.3:
                k = r.random()
                if k < 0.2:
                    fw.lit(",")
                    self.table_ref(fw, d, scope)
                elif k < 0.3:
                    fw.kw("CROSS")
                    fw.kw("JOIN")
                    self.table_ref(fw, d, scope)
                else:
                    jt = r.choice([[], ["INNER"], ["LEFT"], ["LEFT", "OUTER"], ["RIGHT"],
                                   ["RIGHT", "OUTER"], ["FULL"], ["FULL", "OUTER"]])
                    for x in jt:
                        fw.kw(x)
                    fw.kw("JOIN")
                    self.table_ref(fw, d, scope)
                    if r.random() < 0.85:
                        fw.kw("ON")
                        self.bool_expr(fw, scope, d)
                    else:
                        fw.kw("USING")
                        fw.lit("(")
                        t = scope[-1][0] if scope[-1][0] is not None else 0
                        fw.lit(r.choice(self.s.columns[t]))
                        fw.lit(")")
        else:
            scope.append((self.tname(), None))
        if r.random() < 0.12:
            w.lit("*")
        else:
            for i in range(r.randint(1, 4)):
                if i:
                    w.lit(",")
                k = r.random()
                if k < 0.05 and scope[0][1] is not None:
                    w.lit(scope[0][1])
                    w.lit(".")
                    w.lit("*")
                    continue
                if k < 0.08 and scope[0][0] is not None:
                    w.lit(self.s.tables[scope[0][0]])
                    w.lit(".")
                    w.lit("*")
                    continue
                self.value(w, scope, d)
                k2 = r.random()
                if k2 < 0.15:
                    w.kw("AS")
                    w.lit(self.alias())
                elif k2 < 0.2:
                    w.lit(self.alias())
        w.out.extend(fw.out)
        if has_from and r.random() < 0.7:
            w.kw("WHERE")
            self.bool_expr(w, scope, d)
        if has_from and r.random() < 0.15:
            w.kw("GROUP")
            w.kw("BY")
            self.value(w, scope, d)
            for _ in range(r.randint(0, 2)):
                w.lit(",")
                self.value(w, scope, d)
            if r.random() < 0.4:
                w.kw("HAVING")
                self.bool_expr(w, scope, d)
        return scope

    def query_stmt(self, w, d):
        r = self.r
        if d < self.maxd and r.random() < 0.1:
            w.kw("WITH")
            if r.random() < 0.2:
                w.kw("RECURSIVE")
            for i in range(r.randint(1, 2)):
                if i:
                    w.lit(",")
                w.lit(self.alias())
                if r.random() < 0.3:
                    w.lit("(")
                    w.lit(r.choice(self.s.columns[self.tname()]))
                    w.lit(")")
                w.kw("AS")
                w.lit("(")
                self.query_stmt(w, d + 1)
                w.lit(")")
        scope = self.select_core(w, d)
        while r.random() < 0.08:
            op = r.random()
            if op < 0.4:
                w.kw("UNION")
            elif op < 0.6:
                w.kw("UNION")
                w.kw("ALL")
            elif op < 0.8:
                w.kw("INTERSECT")
            else:
                w.kw("EXCEPT")
            scope = self.select_core(w, d)
        if r.random() < 0.25:
            w.kw("ORDER")
            w.kw("BY")
            for i in range(r.randint(1, 2)):
                if i:
                    w.lit(",")
                self.value(w, scope, d)
                c = r.random()
                if c < 0.3:
                    w.kw("ASC")
                elif c < 0.5:
                    w.kw("DESC")
                if r.random() < 0.1:
                    w.kw("NULLS")
                    w.kw(r.choice(["FIRST", "LAST"]))
        if r.random() < 0.25:
            w.kw("LIMIT")
            w.lit(str(r.randint(1, 1000)))
            if r.random() < 0.3:
                w.kw("OFFSET")
                w.lit(str(r.randint(0, 1000)))

    # -- periodic long sentences (flatness with the position isolated)
    def periodic_sentence(self, depth, n_preds=4):
        """(header, block): SELECT .. WHERE <depth nested parens / IN
        subqueries>, then a block of n_preds simple predicates, each followed
        by AND, meant to be repeated; single spaces, fixed keyword case."""
        r = self.r
        t = self.tname()
        cols = lambda: r.choice(self.s.columns[t])
        head = ["SELECT", cols(), "FROM", self.s.tables[t], "WHERE"]
        for lvl in range(depth):
            if lvl % 2 == 0:
                head.append("(")
            else:
                head += [cols(), "IN", "("]
                t = self.tname()
                head += ["SELECT", cols(), "FROM", self.s.tables[t], "WHERE"]
        block = []
        for i in range(n_preds):
            c = cols()
            kind = i % 4
            if kind == 0:
                block += [c, "=", str(r.randint(0, 9999))]
            elif kind == 1:
                block += [c, "IS", "NULL"]
            elif kind == 2:
                block += [c, "IN", "(", str(r.randint(0, 99)), ",", str(r.randint(0, 99)), ")"]
            else:
                block += [c, "<>", "'" + "".join(r.choice("abcdefgh") for _ in range(4)) + "'"]
            block.append("AND")
        return " ".join(head) + " ", " ".join(block) + " "

    # -- long sentences with controlled nesting (position / depth stress)
    def long_sentence(self, depth, min_bytes):
        """SELECT .. WHERE <depth nested parens / IN-subqueries> <long AND/OR
        chain of simple predicates> <closers> ;  -- about min_bytes long."""
        r = self.r
        w = _SqlWriter(r)
        t = self.tname()
        w.kw("SELECT")
        w.lit(r.choice(self.s.columns[t]))
        w.kw("FROM")
        w.lit(self.s.tables[t])
        w.kw("WHERE")
        closers = []
        scope = [(t, None)]
        for lvl in range(depth):
            if lvl % 2 == 0:
                w.lit("(")
                closers.append(")")
            else:
                w.lit(r.choice(self.s.columns[t]))
                w.kw("IN")
                w.lit("(")
                t = self.tname()
                scope = [(t, None)]
                w.kw("SELECT")
                w.lit(r.choice(self.s.columns[t]))
                w.kw("FROM")
                w.lit(self.s.tables[t])
                w.kw("WHERE")
                closers.append(")")
        body = _SqlWriter(r)
        first = True
        total = 0
        while total < min_bytes:
            if not first:
                body.kw("AND" if r.random() < 0.7 else "OR")
            first = False
            mark = len(body.out)
            c = r.choice(self.s.columns[scope[0][0]])
            body.lit(c)
            k = r.random()
            if k < 0.6:
                body.lit(r.choice(["=", "<>", "<", "<=", ">", ">="]))
                body.lit(str(r.randint(0, 9999)) if r.random() < 0.7 else _string_lit(r))
            elif k < 0.8:
                body.kw("IS")
                body.kw("NULL")
            else:
                body.kw("IN")
                body.lit("(")
                body.lit(str(r.randint(0, 99)))
                body.lit(",")
                body.lit(str(r.randint(0, 99)))
                body.lit(")")
            total += sum(len(x) + 1 for x in body.out[mark:])
        w.out.extend(body.out)
        for cl in reversed(closers):
            w.lit(cl)
        w.lit(";")
        return w.text()
