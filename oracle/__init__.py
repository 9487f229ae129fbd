"""Python access to the CPU oracle (ctypes over liboracle.so).

TEST INFRASTRUCTURE ONLY: imported by the test suite, the package smoke check
and the benchmark's CPU-baseline leg.  The product path never imports it.
"""

import ctypes
import os
import subprocess
from pathlib import Path

import numpy as np

HERE = Path(__file__).resolve().parent
LIB = HERE / "liboracle.so"


def build(verbose=False):
    """Compile oracle.cpp into liboracle.so (g++, OpenMP)."""
    cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared", "-Wall",
           "-o", str(LIB) + ".tmp", str(HERE / "oracle.cpp")]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(str(LIB) + ".tmp", LIB)


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not LIB.exists():
            raise RuntimeError(f"{LIB} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(str(LIB))
        c_void_p, c_char_p, c_int, c_size_t = (ctypes.c_void_p, ctypes.c_char_p, ctypes.c_int,
                                               ctypes.c_size_t)
        L.oracle_grammar_new.restype = c_void_p
        L.oracle_grammar_new.argtypes = [c_char_p, c_char_p, c_char_p, c_int]
        L.oracle_grammar_free.argtypes = [c_void_p]
        L.oracle_num_terminals.argtypes = [c_void_p]
        L.oracle_terminal_name.restype = c_char_p
        L.oracle_terminal_name.argtypes = [c_void_p, c_int]
        L.oracle_lexicon_new.restype = c_void_p
        L.oracle_lexicon_new.argtypes = [c_void_p, c_int, ctypes.POINTER(c_char_p),
                                         ctypes.POINTER(c_char_p), c_char_p, c_int]
        L.oracle_lexicon_free.argtypes = [c_void_p]
        L.oracle_vocab_new.restype = c_void_p
        L.oracle_vocab_new.argtypes = [c_void_p, c_void_p, c_int, c_void_p, c_int, ctypes.c_int32]
        L.oracle_vocab_free.argtypes = [c_void_p]
        L.oracle_mask.argtypes = [c_void_p, c_void_p, c_void_p, c_char_p, c_size_t, c_int,
                                  c_void_p, c_int, c_void_p, c_void_p, c_void_p, c_int]
        for f in (L.oracle_viable, L.oracle_member):
            f.argtypes = [c_void_p, c_void_p, c_char_p, c_size_t]
        L.oracle_allowed.argtypes = [c_void_p, c_void_p, c_char_p, c_size_t, c_void_p]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    pass


class Grammar:
    def __init__(self, text, drop=()):
        err = ctypes.create_string_buffer(512)
        h = lib().oracle_grammar_new(text.encode(), ",".join(drop).encode(), err, 512)
        if not h:
            raise OracleError(err.value.decode())
        self.h = h
        self._free = lib().oracle_grammar_free  # kept: module globals may be gone at exit
        self.T = lib().oracle_num_terminals(h)
        self.terminals = [lib().oracle_terminal_name(h, i).decode() for i in range(self.T)]

    def __del__(self):
        if getattr(self, "h", None):
            self._free(self.h)
            self.h = None


class Lexicon:
    def __init__(self, grammar, cats):
        names = list(cats)
        err = ctypes.create_string_buffer(512)
        arr_n = (ctypes.c_char_p * max(1, len(names)))(*[n.encode() for n in names])
        arr_w = (ctypes.c_char_p * max(1, len(names)))(
            *["\n".join(cats[n]).encode() for n in names])
        h = lib().oracle_lexicon_new(grammar.h, len(names), arr_n, arr_w, err, 512)
        if not h:
            raise OracleError(err.value.decode())
        self.h = h
        self._free = lib().oracle_lexicon_free

    def __del__(self):
        if getattr(self, "h", None):
            self._free(self.h)
            self.h = None


class Vocab:
    def __init__(self, spellings, specials=(), eos_id=-1):
        self.V = len(spellings)
        offs = np.zeros(self.V + 1, dtype=np.uint64)
        offs[1:] = np.cumsum([len(t) for t in spellings], dtype=np.uint64)
        data = np.frombuffer(b"".join(spellings) + b"\0", dtype=np.uint8).copy()
        sp = np.asarray(list(specials) or [0], dtype=np.int32)
        self.h = lib().oracle_vocab_new(data.ctypes.data, offs.ctypes.data, self.V,
                                        sp.ctypes.data, len(specials), eos_id)
        self._free = lib().oracle_vocab_free

    def __del__(self):
        if getattr(self, "h", None):
            self._free(self.h)
            self.h = None


class Oracle:
    """Grammar + one lexicon + vocabulary: the mask of Definition 4."""

    def __init__(self, grammar_text, drop=(), lexicon=None, vocab=(), specials=(), eos_id=-1):
        self.grammar = Grammar(grammar_text, drop)
        self.lexicon = Lexicon(self.grammar, lexicon) if lexicon else None
        self.vocab = Vocab(list(vocab), specials, eos_id) if vocab else None
        self.V = len(vocab)

    def _lex(self, lexicon):
        if lexicon is None:
            lexicon = self.lexicon
        return lexicon.h if lexicon is not None else None

    def mask(self, w, mode=1, tokens=None, nthreads=0, lexicon=None):
        """(words uint32[W], eos_ok) for all tokens, or (bits uint8[n], eos_ok)
        for the listed token ids."""
        eos = ctypes.c_int32(0)
        if tokens is None:
            out = np.zeros((self.V + 31) // 32, dtype=np.uint32)
            lib().oracle_mask(self.grammar.h, self._lex(lexicon), self.vocab.h, w, len(w), mode,
                              None, 0, out.ctypes.data, None, ctypes.byref(eos), nthreads)
            return out, int(eos.value)
        ids = np.ascontiguousarray(tokens, dtype=np.int32)
        bits = np.zeros(len(ids), dtype=np.uint8)
        lib().oracle_mask(self.grammar.h, self._lex(lexicon), self.vocab.h, w, len(w), mode,
                          ids.ctypes.data, len(ids), None, bits.ctypes.data, ctypes.byref(eos),
                          nthreads)
        return bits, int(eos.value)

    def viable(self, w, lexicon=None):
        return bool(lib().oracle_viable(self.grammar.h, self._lex(lexicon), w, len(w)))

    def member(self, w, lexicon=None):
        return bool(lib().oracle_member(self.grammar.h, self._lex(lexicon), w, len(w)))

    def allowed(self, w, lexicon=None):
        out = np.zeros(self.grammar.T, dtype=np.uint8)
        ok = lib().oracle_allowed(self.grammar.h, self._lex(lexicon), w, len(w), out.ctypes.data)
        return bool(ok), {self.grammar.terminals[i] for i in range(self.grammar.T) if out[i]}


def from_workload(wl, slot=0):
    """An Oracle for a workload object (see the workloads package)."""
    from workloads import grammar_text
    return Oracle(grammar_text(wl.grammar), wl.drop, wl.lexicons[slot] or None, wl.vocab,
                  wl.specials, wl.eos_id)
