"""The warm path (grid_mask_warm: cached context-independent words, live
context-dependent verdicts) and its cross-family tier T2 on the GPU, through
the C ABI.  Every mask is compared bit for bit with the cold mask of the same
rows (cache-on equals cache-off), and with the oracle where it says so; hits
are confirmed by the cache's state words (a hit publishes nothing new).

* T1 and T2 with genN on random LALR(1) grammars with their own
  vocabularies: warm equals cold, inserting then hitting.
* T1: the benchmark's DML batches, missed then hit; configurations that
  differ only below the top of the stack share an entry; decode loops with
  the device advance, warm masks against cold ones and the oracle each step.
* T2: two role projections of one dialect share entries (the family key);
  numeric remainders of different bytes share an entry under the genN normal
  form, identifier remainders (the lexicon-visibility guard fails) do not;
  one prefix on two schemas gets two entries (the schema fingerprint scopes
  lexicon-bearing producers).
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import grammar_text, make_workload  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    pkg.lib()
    return pkg


def _states(grid, cache):
    stride = 96 + (4 * grid.W + 15) // 16 * 16
    return cache.cpu().numpy().reshape(-1, stride)[:, :4].copy().view(np.uint32)[:, 0]


def _published(grid, cache):
    st = _states(grid, cache)
    return int((st == 2).sum()), int((st == 1).sum())


def _both(G, grid, prefixes, slots, cache, flags):
    cfgs, pool = grid.configs(prefixes, slots)
    c, p = grid.configs_to_device(cfgs, pool)
    B = len(prefixes)
    cold = grid.mask(c, p, B)
    warm = grid.mask_warm(c, p, B, cache, flags)
    torch.cuda.synchronize()
    cold = [x.cpu().numpy() for x in cold]
    warm = [x.cpu().numpy() for x in warm]
    for a, b, what in zip(cold, warm, ("mask", "eos", "status")):
        assert np.array_equal(a, b), what
    assert (warm[2] == 0).all()
    return warm


def test_t1_dml_batches_miss_then_hit(G, oracle_mod):
    wl = make_workload(3, n_batches=2)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    cache = grid.new_ci_cache(1024)
    o = oracle_mod.from_workload(wl)
    for bi, rows in enumerate(wl.batches()):
        prefixes = [wl.prefixes[j] for j in rows]
        slots = [sm[wl.slots[j]] for j in rows]
        before = _published(grid, cache)
        m, e, _ = _both(G, grid, prefixes, slots, cache, G.grid.CI_LOOKUP | G.grid.CI_INSERT)  # misses insert
        after = _published(grid, cache)
        assert after[1] == 0 and after[0] > before[0], (before, after)
        _both(G, grid, prefixes, slots, cache, G.grid.CI_LOOKUP | G.grid.CI_INSERT)           # hits
        assert _published(grid, cache) == after
        got = m.view(np.uint32)
        for r, w in enumerate(prefixes):
            want, want_eos = o.mask(w, mode=1)
            assert np.array_equal(got[r], want), (bi, r)
            assert int(e[r]) == want_eos


@pytest.mark.parametrize("tier", ["t1", "t2_genn"])
def test_warm_equals_cold_on_random_grammars(G, oracle_mod, tier):
    """16 random LALR(1) grammars (workloads.randgram, half of them with
    lexicon categories), each with its own vocabulary and a fresh cache: two
    batches of sampled prefixes (the second sharing keys with the first where
    their rows agree on scan state, remainder and allowed set) run warm twice
    each, first inserting then hitting; every warm mask equals the cold one,
    and the first batch's masks the oracle's.  With T2 the keys also take
    the family fingerprint and the genN normal form of the remainder."""
    from workloads.randgram import RandomGrammar, random_prefixes, random_vocab
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT
    if tier == "t2_genn":
        flags |= G.grid.CI_FAMILY | G.grid.CI_GENN
    n_done = seed = 0
    while n_done < 16:
        rg = RandomGrammar(2000 + seed)
        seed += 1
        assert seed < 300, "too few random grammars compile"
        words = sorted({w for ws in (rg.lexicon or {}).values() for w in ws})
        vocab, specials, eos_id = random_vocab(rg.seed, rg.alphabet(), words=words)
        try:
            grid = G.Grid(rg.text(), (), vocab, specials, eos_id)
        except G.GridError as e:
            assert "GRID_E_LALR_CONFLICT" in str(e), (rg.seed, str(e))
            continue
        slot = grid.add_lexicon(rg.lexicon) if rg.lexicon else 0
        grid.to_device("cuda")
        print(f"random grammar seed {rg.seed}: {tier} lexicon={rg.lexicon is not None}", flush=True)
        cache = grid.new_ci_cache(256)
        o = oracle_mod.Oracle(rg.text(), (), rg.lexicon, vocab, specials, eos_id)
        for half in range(2):
            prefixes = random_prefixes(rg, rg.seed * 2 + half, 16)
            m, e, _ = _both(G, grid, prefixes, [slot] * len(prefixes), cache, flags)   # inserts
            n1 = _published(grid, cache)
            _both(G, grid, prefixes, [slot] * len(prefixes), cache, flags)            # hits
            assert _published(grid, cache) == n1
            if half == 0:
                got = m.view(np.uint32)
                for r, w in enumerate(prefixes):
                    want, want_eos = o.mask(w, mode=1)
                    assert np.array_equal(got[r], want) and int(e[r]) == int(want_eos), (rg.seed, w)
        n_done += 1


def test_t1_entry_shared_by_stacks_that_differ_below_the_top(G):
    """The key holds A(sigma), not the stack: configurations whose stacks
    differ below the top but agree on the scan state, the remainder and the
    allowed set share one entry, while their context-dependent tokens are
    still judged against each one's own stack."""
    wl = make_workload(3, rows=1)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    s = sm[wl.slots[0]]
    t, c = wl.meta["schema"].tables[0], wl.meta["schema"].columns[0][0]
    base = f"select {c} from {t} where {c} = 1 and ".encode()
    deep = f"select {c} from {t} where ({c} = 1 and ".encode()
    cache = grid.new_ci_cache(256)
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT
    _both(G, grid, [base], [s], cache, flags)
    n1 = _published(grid, cache)
    _both(G, grid, [deep], [s], cache, flags)
    assert _published(grid, cache) == n1      # the deeper stack hit the entry
    _both(G, grid, [base, deep, base + b"(", deep + b"("], [s] * 4, cache, flags)


@pytest.mark.parametrize("k", [2, 3])
def test_t1_warm_decode_loop_equals_cold_and_oracle(G, oracle_mod, k):
    wl = make_workload(k, rows=16 if k == 2 else 32)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    o = oracle_mod.from_workload(wl)
    B = len(wl.prefixes)
    slots = [sm[s] for s in wl.slots]
    rng = np.random.default_rng(9100 + k)
    prefixes = list(wl.prefixes)
    cfgs, pool = grid.configs(prefixes, slots)
    c, p = grid.configs_to_device(cfgs, pool)
    cache = grid.new_ci_cache(4096)
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT
    hits = 0
    for step in range(8):
        before = _published(grid, cache)[0]
        m, e, s = grid.mask(c, p, B)
        mw, ew, sw = grid.mask_warm(c, p, B, cache, flags)
        torch.cuda.synchronize()
        assert np.array_equal(m.cpu().numpy(), mw.cpu().numpy()), step
        assert np.array_equal(e.cpu().numpy(), ew.cpu().numpy()) and (sw.cpu().numpy() == 0).all()
        hits += B - (_published(grid, cache)[0] - before)
        got = mw.cpu().numpy().view(np.uint32)
        for r in range(B):
            want, _ = o.mask(prefixes[r], mode=1)
            assert np.array_equal(got[r], want), (step, r)
        bits = np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
        toks = np.zeros(B, np.int32)
        for r in range(B):
            allowed = np.flatnonzero(bits[r])
            allowed = allowed[allowed != wl.eos_id]
            toks[r] = rng.choice(allowed)
        c, p2, st = grid.accept(c, p, torch.from_numpy(toks).cuda(), B, 1024)
        p = p2.view(torch.int16)
        torch.cuda.synchronize()
        assert (st.cpu().numpy() == 0).all()
        for r in range(B):
            prefixes[r] += wl.vocab[toks[r]]
    print(f"workload {k}: {hits} of {8 * B} warm rows served by cached words", flush=True)


def test_t2_roles_share_the_family_entries(G):
    wl = make_workload(3, rows=1)
    lex = wl.lexicons[0]
    ro = G.Grid(grammar_text("sql_dml"), wl.drop, wl.vocab, wl.specials, wl.eos_id)
    full = G.Grid(grammar_text("sql_dml"), [], wl.vocab, wl.specials, wl.eos_id)
    s_ro, s_full = ro.add_lexicon(lex), full.add_lexicon(lex)
    ro.to_device("cuda")
    full.to_device("cuda")
    t, c = wl.meta["schema"].tables[0], wl.meta["schema"].columns[0][0]
    prefixes = [f"select {c} from {t} where {c} = ".encode(), f"select {c}, ".encode(), b"select 1 + 2"]
    cache = ro.new_ci_cache(256)
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT | G.grid.CI_FAMILY
    _both(G, ro, prefixes, [s_ro] * 3, cache, flags)
    n1 = _published(ro, cache)
    _both(G, full, prefixes, [s_full] * 3, cache, flags)
    assert _published(ro, cache) == n1        # the other role hit every entry
    # the per-handle key (T1) does not share across roles
    cache1 = ro.new_ci_cache(256)
    _both(G, ro, prefixes, [s_ro] * 3, cache1, G.grid.CI_LOOKUP | G.grid.CI_INSERT)
    m1 = _published(ro, cache1)
    _both(G, full, prefixes, [s_full] * 3, cache1, G.grid.CI_LOOKUP | G.grid.CI_INSERT)
    assert _published(ro, cache1)[0] == 2 * m1[0]


def test_t2_genn_normal_form_and_the_lexicon_guard(G):
    wl = make_workload(3, rows=1)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    s = sm[wl.slots[0]]
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT | G.grid.CI_FAMILY | G.grid.CI_GENN
    cache = grid.new_ci_cache(256)
    _both(G, grid, [b"select 12"], [s], cache, flags)
    n1 = _published(grid, cache)
    _both(G, grid, [b"select 34567"], [s], cache, flags)   # same scan state, other bytes: shared
    assert _published(grid, cache) == n1
    t = wl.meta["schema"].tables
    _both(G, grid, [f"select * from {t[0][:3]}".encode()], [s], cache, flags)
    n2 = _published(grid, cache)
    assert n2[0] == n1[0] + 1
    other = next(x for x in t if x[:3] != t[0][:3] and len(x) >= 3)
    _both(G, grid, [f"select * from {other[:3]}".encode()], [s], cache, flags)
    assert _published(grid, cache)[0] == n2[0] + 1          # lexicon in play: raw remainder kept
    # without genN the numeric remainders do not share
    plain = grid.new_ci_cache(256)
    f2 = G.grid.CI_LOOKUP | G.grid.CI_INSERT | G.grid.CI_FAMILY
    _both(G, grid, [b"select 12"], [s], plain, f2)
    _both(G, grid, [b"select 34567"], [s], plain, f2)
    assert _published(grid, plain)[0] == 2


def test_t2_schema_fingerprint_scopes_entries(G):
    """One prefix on two schemas: two entries, each schema's own mask."""
    wl = make_workload(5, rows=2)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    flags = G.grid.CI_LOOKUP | G.grid.CI_INSERT | G.grid.CI_FAMILY | G.grid.CI_GENN
    cache = grid.new_ci_cache(256)
    pre = [b"SELECT * FROM "]
    m0, _, _ = _both(G, grid, pre, [sm[0]], cache, flags)
    n1 = _published(grid, cache)
    m1, _, _ = _both(G, grid, pre, [sm[1]], cache, flags)
    assert _published(grid, cache)[0] == n1[0] + 1
    assert not np.array_equal(m0, m1)
    _both(G, grid, pre * 2, [sm[0], sm[1]], cache, flags)      # both hit their own entry
    assert _published(grid, cache)[0] == n1[0] + 1
