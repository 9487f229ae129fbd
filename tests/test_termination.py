"""Termination machinery (section 5, Proposition 9, mode 1) on the host,
checked by the oracle.

* grid_complete: for prefixes of every workload -- the 16,000-token
  sentences' deepest configurations included -- the returned tokens complete
  the prefix into a sentence of L, and every intermediate output is a viable
  prefix (a masked decoder could have produced them); pending identifiers are
  finished with words of the row's own schema.
* The reserve trigger in a mode-1 decode loop: sampling from the oracle's
  masks under a token budget, the loop writes the completion and the
  end-of-sequence token once budget <= reserve + safety; every stop is a
  sentence of L within the budget.
* Errors: a non-viable prefix, and a budget smaller than the completion.
"""

import random

import numpy as np
import pytest

from workloads import make_workload


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    pkg.lib()
    return pkg


def _text(wl, toks):
    return b"".join(wl.vocab[t] for t in toks)


@pytest.mark.parametrize("k", [1, 2, 3, 5])
def test_completions_are_sentences_and_every_step_is_viable(G, oracle_mod, k):
    wl = make_workload(k, rows=24 if k != 5 else 6)
    grid, slots = G.from_workload(wl)
    oracles = {}
    for j, w in enumerate(wl.prefixes):
        if wl.slots[j] not in oracles:
            oracles[wl.slots[j]] = oracle_mod.from_workload(wl, slot=wl.slots[j])
        o = oracles[wl.slots[j]]
        toks = grid.complete(w, slots[wl.slots[j]])
        assert o.member(w + _text(wl, toks)), (k, j, w[-40:], _text(wl, toks))
        cur = w
        for t in toks:
            cur += wl.vocab[t]
            assert o.viable(cur), (k, j, cur[-40:])


def test_completions_of_deep_long_prefixes(G, oracle_mod):
    """The deepest configurations of the 16,000-token workload (nesting up to
    128): the completion closes every open construct."""
    wl = make_workload(4, rows=1)
    grid, slots = G.from_workload(wl)
    o = oracle_mod.from_workload(wl)
    cells = wl.meta["cells"]
    for j, w in enumerate(wl.prefixes):
        if cells[j][0] != 1000:
            continue
        toks = grid.complete(w, slots[0])
        assert o.member(w + _text(wl, toks)), (cells[j], _text(wl, toks)[-60:])
        if cells[j][1] == 128:
            assert len(toks) >= 64  # some tokens close more than one level


def test_reserve_trigger_mode1_decode_loop(G, oracle_mod):
    """Mode-1 decode loop: tokens sampled from the exact masks until the
    remaining budget reaches the prefix's reserve plus a safety margin, then
    the completion and the end-of-sequence token are written."""
    wl = make_workload(2, rows=8)
    grid, slots = G.from_workload(wl)
    o = oracle_mod.from_workload(wl)
    r = random.Random(9300)
    budget, safety = 40, 12
    stops = 0
    for j, w0 in enumerate(wl.prefixes):
        w, used = w0, 0
        while True:
            reserve = grid.complete(w, slots[0])
            if budget - used <= len(reserve) + safety:
                w += _text(wl, reserve)
                used += len(reserve)
                break
            words, eos = o.mask(w, mode=1)
            bits = np.unpackbits(words.view(np.uint8), bitorder="little")[:wl.V]
            allowed = [t for t in np.flatnonzero(bits).tolist() if t != wl.eos_id]
            if eos and r.random() < 0.2:
                break
            t = r.choice(allowed)
            w += wl.vocab[t]
            used += 1
        assert used <= budget, (j, used)
        assert o.member(w), (j, w[-60:])
        stops += 1
    assert stops == len(wl.prefixes)


def test_completion_errors(G):
    wl = make_workload(3, rows=1)
    grid, slots = G.from_workload(wl)
    with pytest.raises(G.GridError) as ei:
        grid.complete(b"select from from", slots[0])
    assert ei.value.code == -8
    w = b"select (((((1"
    need = len(grid.complete(w, slots[0]))
    assert need >= 2
    with pytest.raises(G.GridError) as ei:
        grid.complete(w, slots[0], max_tokens=need - 1)
    assert ei.value.code == -11
