"""The per-row persistent stack arena and the rolling configuration hash on
the GPU (grid_accept_inplace, grid_stack_hash, the hash-keyed mask cache),
through the C ABI.

* grid_stack_hash on the device equals the host hash (itself pinned to
  hashlib's BLAKE2b on the CPU) on workload stacks, deep ones included.
* In-place decode loops: each row's stack lives in its own region of the pool
  and is advanced in place; after every step the configuration and stack equal
  the host advance of the extended prefix, the kept rolling hashes equal the
  host hash of the new stack (only the rewritten entries were recomputed),
  and the mask of the advanced configuration equals the oracle's.
* The same decode loops on random LALR(1) grammars with their own
  vocabularies (half of them with lexicon categories), ending rows that can
  only stop with the end-of-sequence token.
* A refused token leaves the row's configuration, stack and hashes untouched.
* The mask cache keyed by H(top) gives the cold masks (cache-on equals
  cache-off), and a repeated configuration is a hit.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import make_workload  # noqa: E402

pytestmark = pytest.mark.gpu

CAP = 1024


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    pkg.lib()
    return pkg


def _regions(G, grid, prefixes, slots, cap=CAP):
    """Configurations with row b's stack at pool[b * cap ..]."""
    cfgs, pool = grid.configs(prefixes, slots)
    region = np.zeros(len(prefixes) * cap, dtype=np.uint16)
    for b in range(len(prefixes)):
        off, d = int(cfgs["stk_off"][b]), int(cfgs["stk_depth"][b])
        region[b * cap:b * cap + d] = pool[off:off + d]
        cfgs["stk_off"][b] = b * cap
    return cfgs, region


def _host_hashes(grid, cfgs, pool):
    out = {}
    for b in range(len(cfgs)):
        off, d = int(cfgs["stk_off"][b]), int(cfgs["stk_depth"][b])
        out[b] = grid.stack_hash_host(pool[off:off + d])
    return out


def test_device_stack_hash_equals_host(G):
    for k, kw in ((3, dict(rows=32)), (4, dict(rows=2))):
        wl = make_workload(k, **kw)
        grid, slots = G.from_workload(wl)
        grid.to_device("cuda")
        rows = list(range(0, len(wl.prefixes), max(1, len(wl.prefixes) // 32)))[:32]
        cfgs, pool = grid.configs([wl.prefixes[j] for j in rows], [slots[wl.slots[j]] for j in rows])
        c, p = grid.configs_to_device(cfgs, pool)
        h = grid.stack_hash(c, p, len(rows))
        torch.cuda.synchronize()
        got = h.cpu().numpy().view(np.uint64)
        want = _host_hashes(grid, cfgs, pool)
        for b in range(len(rows)):
            off, d = int(cfgs["stk_off"][b]), int(cfgs["stk_depth"][b])
            assert np.array_equal(got[off:off + d], want[b]), (k, b)
        assert int(cfgs["stk_depth"].max()) > (300 if k == 4 else 3)


@pytest.mark.parametrize("k", [2, 3])
def test_inplace_decode_loop_matches_host_and_oracle(G, oracle_mod, k):
    wl = make_workload(k, rows=16 if k == 2 else 32)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    o = oracle_mod.from_workload(wl)
    B = len(wl.prefixes)
    slots = [slot_map[s] for s in wl.slots]
    rng = np.random.default_rng(7100 + k)
    prefixes = list(wl.prefixes)
    cfgs, region = _regions(G, grid, prefixes, slots)
    c, p = grid.configs_to_device(cfgs, region)
    h = grid.stack_hash(c, p, B)
    cache = grid.new_cache(4096)
    for step in range(8):
        m, e, s = grid.mask(c, p, B)
        mc, ec, sc = grid.mask(c, p, B, cache=cache, stack_hash=h)   # keyed by H(top)
        torch.cuda.synchronize()
        assert np.array_equal(m.cpu().numpy(), mc.cpu().numpy()) and np.array_equal(e.cpu().numpy(), ec.cpu().numpy())
        assert np.array_equal(s.cpu().numpy(), sc.cpu().numpy())
        bits = np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
        toks = np.zeros(B, np.int32)
        for r in range(B):
            allowed = np.flatnonzero(bits[r])
            allowed = allowed[allowed != wl.eos_id]
            toks[r] = rng.choice(allowed)
        st = grid.accept_inplace(c, p, torch.from_numpy(toks).cuda(), B, CAP, stack_hash=h)
        torch.cuda.synchronize()
        assert (st.cpu().numpy() == G.ROW_OK).all(), (step, st.cpu().numpy().tolist())
        for r in range(B):
            prefixes[r] = prefixes[r] + wl.vocab[toks[r]]
        got = c.cpu().numpy().view(G.CONFIG_DTYPE)
        pool = p.cpu().numpy().view(np.uint16)
        hashes = h.cpu().numpy().view(np.uint64)
        for r in range(B):
            want, stack = grid.config(prefixes[r], slots[r])
            for f in ("q", "lexnode", "flags", "rem_len", "slot"):
                assert int(got[r][f]) == int(want[f]), (step, r, f)
            assert bytes(got[r]["rem_head"]) == bytes(want["rem_head"])
            off, d = int(got[r]["stk_off"]), int(got[r]["stk_depth"])
            assert off == r * CAP and d == len(stack), (step, r)
            assert np.array_equal(pool[off:off + d], stack), (step, r)
            assert np.array_equal(hashes[off:off + d], grid.stack_hash_host(stack)), (step, r)
        m, e, s = grid.mask(c, p, B)
        torch.cuda.synchronize()
        gm = m.cpu().numpy().view(np.uint32)
        for r in range(B):
            want, want_eos = o.mask(prefixes[r], mode=1)
            assert np.array_equal(gm[r], want), (step, r)
            assert int(e[r]) == want_eos
    # a repeated batch hits: nothing new is published
    before = _published(grid, cache)
    mc, _, _ = grid.mask(c, p, B, cache=cache, stack_hash=h)
    grid.mask(c, p, B, cache=cache, stack_hash=h)
    torch.cuda.synchronize()
    mid = _published(grid, cache)
    grid.mask(c, p, B, cache=cache, stack_hash=h)
    torch.cuda.synchronize()
    assert _published(grid, cache) == mid and mid[0] >= before[0]
    # a refused token leaves the rows untouched
    bits = np.unpackbits(mc.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
    toks = np.array([rng.choice(np.flatnonzero(bits[r] == 0)) for r in range(B)], np.int32)
    toks = np.where(toks == wl.eos_id, toks - 1, toks).astype(np.int32)
    before = (c.cpu().numpy().copy(), p.cpu().numpy().copy(), h.cpu().numpy().copy())
    st = grid.accept_inplace(c, p, torch.from_numpy(toks).cuda(), B, CAP, stack_hash=h)
    torch.cuda.synchronize()
    blocked = [r for r in range(B) if not bits[r][toks[r]]]
    assert (st.cpu().numpy()[blocked] == G.ROW_NOT_VIABLE).all()
    after = (c.cpu().numpy(), p.cpu().numpy(), h.cpu().numpy())
    for x, y in zip(before, after):
        assert np.array_equal(x, y)


def _published(grid, cache):
    stride = 64 + (4 * grid.W + 15) // 16 * 16
    states = cache.cpu().numpy().reshape(-1, stride)[:, :4].copy().view(np.uint32)[:, 0]
    return int((states == 2).sum()), int((states == 1).sum())


def test_inplace_decode_loops_on_random_grammars(G, oracle_mod):
    """Decode loops on 16 random LALR(1) grammars (workloads.randgram, half of
    them with lexicon categories), 16 rows each, 6 steps: a token sampled from
    each row's GPU mask is accepted in place; the configuration and stack
    then equal the host advance of the extended prefix, the kept rolling
    hashes the host hash of the new stack, and the new mask the oracle's.  A
    row whose mask allows only the end of sequence takes it and reports
    GRID_ROW_FINISHED, untouched."""
    from workloads.randgram import RandomGrammar, random_prefixes, random_vocab
    n_done = seed = 0
    while n_done < 16:
        rg = RandomGrammar(1000 + seed)
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
        o = oracle_mod.Oracle(rg.text(), (), rg.lexicon, vocab, specials, eos_id)
        prefixes = random_prefixes(rg, rg.seed, 16)
        B = len(prefixes)
        print(f"random grammar seed {rg.seed}: B={B} lexicon={rg.lexicon is not None}", flush=True)
        cfgs, region = _regions(G, grid, prefixes, [slot] * B, cap=256)
        c, p = grid.configs_to_device(cfgs, region)
        h = grid.stack_hash(c, p, B)
        rng = np.random.default_rng(rg.seed)
        for step in range(6):
            m, e, s = grid.mask(c, p, B)
            torch.cuda.synchronize()
            bits = np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :len(vocab)]
            toks = np.zeros(B, np.int32)
            for r in range(B):
                allowed = np.flatnonzero(bits[r])
                rest = allowed[allowed != eos_id]
                assert len(allowed) > 0, (rg.seed, step, prefixes[r])
                toks[r] = rng.choice(rest) if len(rest) else eos_id
            st = grid.accept_inplace(c, p, torch.from_numpy(toks).cuda(), B, 256, stack_hash=h)
            torch.cuda.synchronize()
            st = st.cpu().numpy()
            for r in range(B):
                if toks[r] == eos_id:
                    assert st[r] == G.ROW_FINISHED, (rg.seed, step, r, st[r])
                else:
                    assert st[r] == G.ROW_OK, (rg.seed, step, r, st[r])
                    prefixes[r] = prefixes[r] + vocab[toks[r]]
            got = c.cpu().numpy().view(G.CONFIG_DTYPE)
            pool = p.cpu().numpy().view(np.uint16)
            hashes = h.cpu().numpy().view(np.uint64)
            for r in range(B):
                want, stack = grid.config(prefixes[r], slot)
                for f in ("q", "lexnode", "flags", "rem_len", "slot"):
                    assert int(got[r][f]) == int(want[f]), (rg.seed, step, r, f)
                assert bytes(got[r]["rem_head"]) == bytes(want["rem_head"])
                off, d = int(got[r]["stk_off"]), int(got[r]["stk_depth"])
                assert off == r * 256 and d == len(stack), (rg.seed, step, r)
                assert np.array_equal(pool[off:off + d], stack), (rg.seed, step, r)
                assert np.array_equal(hashes[off:off + d], grid.stack_hash_host(stack)), (rg.seed, step, r)
            m, e, s = grid.mask(c, p, B)
            torch.cuda.synchronize()
            gm, ge = m.cpu().numpy().view(np.uint32), e.cpu().numpy()
            for r in range(B):
                want, want_eos = o.mask(prefixes[r], mode=1)
                assert np.array_equal(gm[r], want) and int(ge[r]) == int(want_eos), (rg.seed, step, prefixes[r])
        n_done += 1


def test_inplace_rejects_rows_outside_their_region(G):
    """A configuration whose stack is not at its row's region is a bad
    configuration; nothing of it is written."""
    wl = make_workload(3, rows=2)
    grid, slots = G.from_workload(wl)
    grid.to_device("cuda")
    cfgs, region = _regions(G, grid, wl.prefixes, [slots[s] for s in wl.slots])
    cfgs["stk_off"][1] = 3
    c, p = grid.configs_to_device(cfgs, region)
    before = c.cpu().numpy().copy()
    vocab = {t: i for i, t in enumerate(wl.vocab)}
    st = grid.accept_inplace(c, p, torch.tensor([vocab[b" "]] * 2, dtype=torch.int32).cuda(), 2, CAP)
    torch.cuda.synchronize()
    assert st.cpu().numpy()[1] == G.ROW_BAD_CONFIG
    assert np.array_equal(c.cpu().numpy()[32:], before[32:])
