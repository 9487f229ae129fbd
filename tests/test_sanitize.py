"""AddressSanitizer + UndefinedBehaviorSanitizer runs of the host C++ on the
CPU: the library's host side (grammar compiler, LALR and lexer construction,
vocabulary and class artifacts, lexicon slots, host advance, rolling hash,
completion writer, compiler error paths) and the oracle, each linked into a
driver of its own (tests/sanitize/) and run on case files written from the
workloads.  Any sanitizer report aborts the driver (no recovery), so a zero
exit status means a clean run.
"""

import shutil
import subprocess
from pathlib import Path

import pytest

from workloads import make_workload
from workloads.configs import GRAMMAR_DIR

ROOT = Path(__file__).resolve().parents[1]
CSRC = ROOT / "paper_2607_11951_amd" / "csrc"
HOST = ["grammar.cpp", "lexer.cpp", "parser.cpp", "artifacts.cpp", "advance.cpp", "complete.cpp", "capi.cpp"]
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1",
       "-std=c++17", "-pthread"]
ENV = {"ASAN_OPTIONS": "detect_leaks=1:abort_on_error=1:allocator_may_return_null=0",
       "UBSAN_OPTIONS": "print_stacktrace=1:halt_on_error=1", "PATH": "/usr/bin:/bin"}


def _compile(out, sources, extra=()):
    cmd = ["g++", *SAN, *extra, *map(str, sources), "-o", str(out)]
    subprocess.run(cmd, check=True, capture_output=True, timeout=900)
    return out


@pytest.fixture(scope="module")
def drivers(tmp_path_factory):
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    d = tmp_path_factory.mktemp("san")
    probe = d / "probe.cpp"
    probe.write_text("int main() { return 0; }\n")
    try:
        _compile(d / "probe", [probe])
    except subprocess.CalledProcessError:
        pytest.skip("the sanitizer runtimes are not installed")
    objs = []
    procs = []
    for s in HOST:
        o = d / (s + ".o")
        procs.append(subprocess.Popen(["g++", *SAN, "-c", str(CSRC / s), "-o", str(o)]))
        objs.append(o)
    assert all(p.wait(timeout=900) == 0 for p in procs)
    host = _compile(d / "host_driver", [ROOT / "tests" / "sanitize" / "host_driver.cpp", *objs])
    oracle = _compile(d / "oracle_driver", [ROOT / "tests" / "sanitize" / "oracle_driver.cpp",
                                            ROOT / "oracle" / "oracle.cpp"], ["-fopenmp"])
    return d, host, oracle


def _write_case(path, grammar, drop, vocab, specials, eos, lexicon, prefixes, n_masks):
    h = lambda b: b.hex() if b else "-"
    lines = [f"G {GRAMMAR_DIR / (grammar + '.grid')}", f"D {','.join(drop) if drop else '-'}", f"E {eos}",
             f"V {len(vocab)}", *[h(v) for v in vocab], f"S {len(specials)} " + " ".join(map(str, specials))]
    if lexicon:
        lines.append(f"L {len(lexicon)}")
        for name, words in lexicon.items():
            lines.append(f"{name} {len(words)}")
            lines += list(words)
    lines += [f"P {len(prefixes)}", *[h(p) for p in prefixes], f"M {n_masks}"]
    path.write_text("\n".join(lines) + "\n")
    return path


def _cases(d):
    out = []
    wl = make_workload(1)
    out.append(_write_case(d / "expr.case", wl.grammar, wl.drop, wl.vocab, wl.specials, wl.eos_id, None,
                           wl.prefixes[:48], 8))
    for k in (2, 3):
        wl = make_workload(k, rows=16)
        # the workload's own grammar and lexicon with a cut vocabulary: every
        # single byte, then the first ids (keywords and identifiers included)
        keep = [t for t in range(min(wl.V, 6000)) if t not in wl.specials]
        vocab = [wl.vocab[t] for t in keep] + [b""]
        out.append(_write_case(d / f"w{k}.case", wl.grammar, wl.drop, vocab, [len(vocab) - 1], len(vocab) - 1,
                               wl.lexicons[wl.slots[0]] or None, wl.prefixes, 4))
    vocab = [bytes([b]) for b in range(256)] + [b"select", b" *", b" from", b" employees", b";", b""]
    out.append(_write_case(d / "crud.case", "crud", ["insert", "update", "delete"], vocab, [len(vocab) - 1],
                           len(vocab) - 1, {"TABLE_NAME": ["employees", "orders"], "COLUMN_NAME": ["id", "name"]},
                           [b"", b"select", b"select * from employees where id = 1", b"select * from emp",
                            b"select * from employees;"], 5))
    return out


def test_host_and_oracle_under_asan_ubsan(drivers):
    d, host, oracle = drivers
    for case in _cases(d):
        for exe in (host, oracle):
            r = subprocess.run([str(exe), str(case)], capture_output=True, text=True, timeout=900, env=ENV)
            assert r.returncode == 0, f"{exe.name} {case.name}: rc={r.returncode}\n{r.stdout}\n{r.stderr[-4000:]}"
            assert "runtime error" not in r.stderr and "AddressSanitizer" not in r.stderr, r.stderr[-4000:]
            print(case.name, r.stdout.strip())
