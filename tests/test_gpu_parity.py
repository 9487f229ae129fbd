"""GPU path (libgrid.so HIP kernels, called through the C ABI) against the CPU
oracle, element by element, bit-exact.

Masks are compared word for word with the oracle's full mask for every row
(checkpoint mode of the oracle, itself checked equal to from-scratch mode on
CPU tests) at every workload's real size and in the launch configuration the
benchmark times; end-of-sequence flags and row status are checked too.  The
apply kernel is compared with torch's CPU masked_fill on fp32 and bf16.
"""

import os
import sys
import time

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import make_workload  # noqa: E402

pytestmark = pytest.mark.gpu


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    pkg.lib()  # raises when libgrid.so is missing: no fallback
    return pkg


def _gpu_masks(G, wl, rows, grid=None, slot_map=None):
    """Runs the GPU path over rows in batches of wl.batch; returns host arrays."""
    if grid is None:
        grid, slot_map = G.from_workload(wl)
        grid.to_device("cuda")
    masks, eos, status = [], [], []
    for i in range(0, len(rows), wl.batch):
        idx = rows[i:i + wl.batch]
        cfgs, pool = grid.configs([wl.prefixes[j] for j in idx], [slot_map[wl.slots[j]] for j in idx])
        c, p = grid.configs_to_device(cfgs, pool)
        m, e, s = grid.mask(c, p, len(idx))
        torch.cuda.synchronize()
        masks.append(m.cpu().numpy().view(np.uint32))
        eos.append(e.cpu().numpy())
        status.append(s.cpu().numpy())
    _gpu_masks.slot_map = slot_map
    return grid, np.concatenate(masks), np.concatenate(eos), np.concatenate(status)


def _oracle_rows(oracle_mod, wl, rows):
    o = oracle_mod.from_workload(wl)
    out, eos = [], []
    lex_cache = {}
    for j in rows:
        lexicon = None
        if len(wl.lexicons) > 1:
            s = wl.slots[j]
            if s not in lex_cache:
                lex_cache[s] = oracle_mod.Lexicon(o.grammar, wl.lexicons[s])
            lexicon = lex_cache[s]
        w, e = o.mask(wl.prefixes[j], mode=1, lexicon=lexicon)
        out.append(w)
        eos.append(e)
    return np.stack(out), np.array(eos, dtype=np.uint8)


def _compare(wl, rows, gm, ge, gs, om, oe, label):
    bad_rows = [r for r in range(len(rows)) if not np.array_equal(gm[r], om[r]) or ge[r] != oe[r]]
    for r in bad_rows[:3]:
        diff = np.nonzero(gm[r] != om[r])[0]
        toks = []
        for w in diff[:4]:
            x = int(gm[r][w]) ^ int(om[r][w])
            toks += [int(w) * 32 + b for b in range(32) if (x >> b) & 1][:3]
        log(f"[{label}] row {rows[r]} prefix={wl.prefixes[rows[r]][-60:]!r} eos gpu={ge[r]} "
            f"oracle={oe[r]} differing tokens {[(t, wl.vocab[t]) for t in toks[:6]]}")
    assert not bad_rows, f"{label}: {len(bad_rows)} rows differ"
    assert (gs == 0).all(), f"{label}: row status {gs}"
    # nothing viable is empty (Proposition 8 with a byte-complete vocabulary)
    assert all(int(om[r].any()) or oe[r] for r in range(len(rows)))


def test_expr_all_configs_one_per_call(G, oracle_mod):
    wl = make_workload(1)
    rows = list(range(len(wl.prefixes)))
    log(f"workload 1: {len(rows)} rows, V={wl.V}, one row per call")
    _, gm, ge, gs = _gpu_masks(G, wl, rows)
    om, oe = _oracle_rows(oracle_mod, wl, rows)
    _compare(wl, rows, gm, ge, gs, om, oe, "expr")


def test_select_subset_batch(G, oracle_mod):
    wl = make_workload(2, n_batches=2)
    rows = list(range(len(wl.prefixes)))
    log(f"workload 2: {len(rows)} rows, V={wl.V}, batch {wl.batch}")
    _, gm, ge, gs = _gpu_masks(G, wl, rows)
    om, oe = _oracle_rows(oracle_mod, wl, rows)
    _compare(wl, rows, gm, ge, gs, om, oe, "select")


def test_dml_full_size_batch(G, oracle_mod):
    """The benchmark's workload and launch shape: B = 32, V = 151,936, all
    eight config batches the benchmark cycles through (256 rows)."""
    wl = make_workload(3, n_batches=8)
    rows = list(range(len(wl.prefixes)))
    log(f"workload 3: {len(rows)} rows, V={wl.V}, batch {wl.batch}")
    t = time.time()
    _, gm, ge, gs = _gpu_masks(G, wl, rows)
    om, oe = _oracle_rows(oracle_mod, wl, rows)
    log(f"  compared in {time.time() - t:.1f}s")
    _compare(wl, rows, gm, ge, gs, om, oe, "dml")


def test_long_sentences_positions_and_depths(G, oracle_mod):
    """16,000-token sentences at the shape the flatness measurement times:
    configurations at 1k / 4k / 16k tokens, nesting depth 1 / 8 / 32 / 128,
    all 32 configurations of every (position, depth) cell as one B = 32 call
    (384 rows; stacks up to several hundred states)."""
    t = time.time()
    wl = make_workload(4)
    rows = list(range(len(wl.prefixes)))
    assert wl.batch == 32 and len(rows) == 384
    log(f"workload 4: {len(rows)} rows (32 per cell, B = 32), V={wl.V}, built in {time.time() - t:.1f}s")
    grid, gm, ge, gs = _gpu_masks(G, wl, rows)
    log(f"  GPU done at {time.time() - t:.1f}s")
    om, oe = _oracle_rows(oracle_mod, wl, rows)
    log(f"  oracle done at {time.time() - t:.1f}s")
    _compare(wl, rows, gm, ge, gs, om, oe, "long")
    sm = _gpu_masks.slot_map
    cfgs, _ = grid.configs([wl.prefixes[j] for j in rows[-32:]], [sm[wl.slots[j]] for j in rows[-32:]])
    log(f"  stack depths at depth-128 cells: {sorted(cfgs['stk_depth'].tolist())}")
    assert cfgs["stk_depth"].max() > 500


def test_long_sentences_position_isolated(G, oracle_mod):
    """The position-isolated 16,000-token workload the flatness measurement
    also times: every configuration of the n = 16,000 cells (32 per depth,
    B = 32, stacks up to several hundred states) against the oracle, and the
    masks at n = 1,000 / 4,000 equal to those at 16,000 row for row (same
    local context, only the position differs)."""
    wl = make_workload(6)
    cells = wl.meta["cells"]
    rows = list(range(len(wl.prefixes)))
    grid, gm, ge, gs = _gpu_masks(G, wl, rows)
    assert (gs == 0).all()
    far = [i for i in rows if cells[i][0] == 16000]
    om, oe = _oracle_rows(oracle_mod, wl, far)
    _compare(wl, far, gm[far], ge[far], gs[far], om, oe, "isolated")
    for d in (1, 8, 32, 128):
        by_pos = {p: [i for i in rows if cells[i][1] == d and cells[i][0] == p] for p in (1000, 4000, 16000)}
        for a, b, c in zip(by_pos[1000], by_pos[4000], by_pos[16000]):
            assert np.array_equal(gm[a], gm[c]) and np.array_equal(gm[b], gm[c]), (d, cells[a], cells[c])


def test_worked_example_section_7_1_on_gpu(G, oracle_mod):
    """The paper's first worked example (section 7.1, the golden fixture)
    through the HIP path: the CRUD grammar under the analyst projection, the
    fixture's schema lexicon, and a vocabulary of the 256 single bytes, the
    fixture's spellings and an end-of-sequence id.  Every printed verdict must
    hold on the GPU mask, and the whole mask must equal the oracle's."""
    import json
    from pathlib import Path
    from workloads import grammar_text
    fx = json.loads((Path(__file__).resolve().parent / "golden" / "worked_example_1.json").read_text())
    spells = sorted({s for c in fx["cases"] for k in ("allowed", "blocked") for s in c.get(k, [])})
    vocab = [bytes([b]) for b in range(256)] + [s.encode() for s in spells if len(s.encode()) > 1] + [b""]
    eos = len(vocab) - 1
    g = G.Grid(grammar_text(fx["grammar"]), fx["drop"], vocab, [eos], eos)
    slot = g.add_lexicon(fx["lexicon"])
    g.to_device("cuda")
    prefixes = [c["prefix"].encode() for c in fx["cases"]]
    cfgs, pool = g.configs(prefixes, [slot] * len(prefixes))
    cd, pd = g.configs_to_device(cfgs, pool)
    m, e, s = g.mask(cd, pd, len(prefixes))
    torch.cuda.synchronize()
    o = oracle_mod.Oracle(grammar_text(fx["grammar"]), fx["drop"], fx["lexicon"], vocab, [eos], eos)
    got = m.cpu().numpy().view(np.uint32)
    ids = {sp: i for i, sp in enumerate(vocab)}
    for i, c in enumerate(fx["cases"]):
        bit = lambda sp: (int(got[i][ids[sp] >> 5]) >> (ids[sp] & 31)) & 1  # noqa: E731
        for sp in c.get("allowed", []):
            assert bit(sp.encode()) == 1, (c["prefix"], sp)
        for sp in c.get("blocked", []):
            assert bit(sp.encode()) == 0, (c["prefix"], sp)
        if "eos" in c:
            assert int(e[i]) == int(c["eos"]), c["prefix"]
        want, want_eos = o.mask(prefixes[i], mode=0)
        assert np.array_equal(got[i], want), c["prefix"]
        assert int(e[i]) == want_eos
    assert (s.cpu().numpy() == 0).all()


def test_cold_schema_batch_and_bf16_apply(G, oracle_mod):
    """256 rows, each with its own freshly generated schema lexicon, then the
    fused -inf fill of bf16 logits [256, 151,936] ~ N(0, 4)."""
    wl = make_workload(5)
    rows = list(range(len(wl.prefixes)))
    log(f"workload 5: {len(rows)} rows / schemas, V={wl.V}")
    t = time.time()
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    log(f"  compile + {len(slot_map)} lexicons + upload: {time.time() - t:.1f}s")
    _, gm, ge, gs = _gpu_masks(G, wl, rows, grid, slot_map)
    om, oe = _oracle_rows(oracle_mod, wl, rows)
    _compare(wl, rows, gm, ge, gs, om, oe, "cold-schema")
    gen = torch.Generator(device="cpu").manual_seed(wl.meta["logits_seed"])
    logits = (torch.randn(len(rows), wl.V, generator=gen) * wl.meta["logits_std"]).to(torch.bfloat16)
    ref = _apply_reference(logits, om, wl.V)
    dev = logits.cuda()
    mask_dev = torch.from_numpy(om.view(np.int32).copy()).cuda()
    G.apply(mask_dev, dev)
    torch.cuda.synchronize()
    assert torch.equal(dev.cpu().view(torch.int16), ref.view(torch.int16))


def _apply_reference(logits, words, V):
    bits = np.unpackbits(words.view(np.uint8), axis=1, bitorder="little")[:, :V].astype(bool)
    out = logits.clone()
    out.masked_fill_(~torch.from_numpy(bits), float("-inf"))
    return out


@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("B,V,pad", [(1, 1, 0), (3, 37, 5), (5, 1024, 0), (2, 151936, 8), (7, 1001, 3)])
def test_apply_bit_exact(G, dtype, B, V, pad):
    g = torch.Generator(device="cpu").manual_seed(B * 1000 + V)
    W = (V + 31) // 32
    words = torch.randint(0, 2 ** 32, (B, W), generator=g, dtype=torch.int64).numpy().astype(np.uint32)
    words[0, :] = 0                                   # a fully masked row
    if B > 1:
        words[1, :] = 0xFFFFFFFF                      # a fully allowed row
    if V % 32:
        words[:, -1] &= (1 << (V % 32)) - 1
    store = (torch.randn(B, V + pad, generator=g) * 2).to(dtype)
    ref = store.clone()
    ref[:, :V] = _apply_reference(store[:, :V].contiguous(), words, V)
    dev = store.cuda()
    view = dev[:, :V]
    G.apply(torch.from_numpy(words.view(np.int32).copy()).cuda(), view)
    torch.cuda.synchronize()
    itype = torch.int16 if dtype == torch.bfloat16 else torch.int32
    assert torch.equal(dev.cpu().view(itype), ref.view(itype))


def test_edge_cases(G, oracle_mod):
    wl = make_workload(3, rows=4)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    prefixes = [b"", b"select", b"select 1;", b"select 1; \n ", b"  ", b"with t1 as (select *"]
    cfgs, pool = grid.configs(prefixes, [slot_map[0]] * len(prefixes))
    c, p = grid.configs_to_device(cfgs, pool)
    m, e, s = grid.mask(c, p, len(prefixes))
    torch.cuda.synchronize()
    o = oracle_mod.from_workload(wl)
    for i, w in enumerate(prefixes):
        ow, oe = o.mask(w, mode=1)
        assert np.array_equal(m[i].cpu().numpy().view(np.uint32), ow), w
        assert int(e[i]) == oe, w
    assert e.cpu().tolist() == [0, 0, 1, 1, 0, 0]
    # a configuration with an out-of-range DFA state is flagged, not walked
    bad = cfgs.copy()
    bad["q"][1] = 60000
    c2, p2 = grid.configs_to_device(bad, pool)
    m2, e2, s2 = grid.mask(c2, p2, len(prefixes))
    torch.cuda.synchronize()
    assert s2.cpu().tolist()[1] == G.ROW_BAD_CONFIG
    assert int(m2[1].abs().sum()) == 0 and s2.cpu().tolist()[0] == 0


def test_gpu_invariants_full_vocab(G):
    """Properties that hold at any size: alias ids carry equal bits; a blocked
    spelling blocks every extension (monotone rejection); specials and padding
    bits are 0."""
    wl = make_workload(3, rows=32)
    rows = list(range(32))
    _, gm, ge, gs = _gpu_masks(G, wl, rows)
    bits = np.unpackbits(gm.view(np.uint8), axis=1, bitorder="little")
    V = wl.V
    assert not bits[:, V:].any()
    specials = [t for t in wl.specials if t != wl.eos_id]
    assert not bits[:, specials].any()
    assert (bits[:, wl.eos_id] == ge).all()
    first = {}
    for t, sp in enumerate(wl.vocab):
        if sp and t not in wl.specials:
            first.setdefault(sp, t)
    for t, sp in enumerate(wl.vocab):
        if sp in first and first[sp] != t:
            assert (bits[:, t] == bits[:, first[sp]]).all()
    by_spelling = {sp: t for sp, t in first.items()}
    for sp, t in list(by_spelling.items())[:20000]:
        if len(sp) > 1 and sp[:-1] in by_spelling:
            parent = by_spelling[sp[:-1]]
            assert not (bits[:, t] & ~bits[:, parent]).any(), sp


def test_gpu_composition_invariant(G):
    """Composition (section 4.1): a token t = p + b whose spelling is another
    token p followed by one byte b is allowed at a configuration exactly when
    p is allowed there and the one-byte token b is allowed after p.  Checked
    on the full DML vocabulary from the GPU masks alone: masks at 8 rows, then
    at those rows advanced by up to 48 allowed parents each (one call)."""
    wl = make_workload(3, rows=32)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    first = {}
    for t, sp in enumerate(wl.vocab):
        if sp and t not in wl.specials:
            first.setdefault(sp, t)
    byte_tok = {b: first[bytes([b])] for b in range(256) if bytes([b]) in first}
    children = {}
    for sp, t in first.items():
        if len(sp) > 1 and sp[:-1] in first and sp[-1] in byte_tok:
            children.setdefault(first[sp[:-1]], []).append((t, byte_tok[sp[-1]]))

    def masks(prefixes, slots):
        cfgs, pool = grid.configs(prefixes, slots)
        c, p = grid.configs_to_device(cfgs, pool)
        m, _, s = grid.mask(c, p, len(prefixes))
        torch.cuda.synchronize()
        assert (s.cpu().numpy() == 0).all()
        return np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")

    rows = list(range(0, 32, 4))
    base = masks([wl.prefixes[j] for j in rows], [sm[wl.slots[j]] for j in rows])
    rng = np.random.default_rng(4100)
    ext, ext_slots, pairs = [], [], []
    for i, j in enumerate(rows):
        parents = [pt for pt in children if base[i, pt]]
        for pt in rng.permutation(parents)[:48].tolist():
            pairs.append((i, pt, len(ext)))
            ext.append(wl.prefixes[j] + wl.vocab[pt])
            ext_slots.append(sm[wl.slots[j]])
    assert len(pairs) >= 8 * 24
    after = masks(ext, ext_slots)
    checked = 0
    for i, pt, e in pairs:
        for t, bt in children[pt]:
            assert base[i, t] == after[e, bt], (rows[i], wl.vocab[pt], wl.vocab[t])
            checked += 1
    # and a blocked parent blocks all its children (monotone rejection)
    for i in range(len(rows)):
        for pt, kids in children.items():
            if not base[i, pt]:
                assert not any(base[i, t] for t, _ in kids)
    log(f"composition: {checked} (token, parent, byte) triples at {len(pairs)} advanced rows")


def test_random_grammars_match_oracle(G, oracle_mod):
    """48 random grammars (workloads.randgram: chains of one-symbol
    productions, empty productions, recursion, nesting, keywords that the
    identifier regex also matches, and in about half of them two lexicon
    categories in its place, every third under a role projection that drops
    one or two labelled alternatives), each with its own vocabulary of 496
    tokens (the lexicon words among them) and 16 sampled prefixes in one
    batch, or 40 for every fourth grammar (two residue row groups): masks,
    end-of-sequence flags and row status bit-exact against the oracle."""
    import random
    from workloads.randgram import RandomGrammar, random_prefixes, random_vocab
    n_done = seed = 0
    while n_done < 48:
        rg = RandomGrammar(seed)
        seed += 1
        assert seed < 600, "too few random grammars compile"
        words = sorted({w for ws in (rg.lexicon or {}).values() for w in ws})
        vocab, specials, eos_id = random_vocab(rg.seed, rg.alphabet(), words=words)
        drop = rg.random_drop(random.Random(rg.seed), 1 + rg.seed % 2) if n_done % 3 == 2 else []
        try:
            grid = G.Grid(rg.text(), drop, vocab, specials, eos_id)
        except G.GridError as e:
            assert "GRID_E_LALR_CONFLICT" in str(e) or "GRID_E_EMPTY_LANGUAGE" in str(e), (rg.seed, str(e))
            continue
        slot = grid.add_lexicon(rg.lexicon) if rg.lexicon else 0
        prefixes = random_prefixes(rg, rg.seed, 40 if n_done % 4 == 3 else 16, drop=drop)
        log(f"random grammar seed {rg.seed}: T={grid.info()['n_terminals']} V={len(vocab)} B={len(prefixes)} "
            f"lexicon={rg.lexicon is not None} drop={drop}")
        grid.to_device("cuda")
        cfgs, pool = grid.configs(prefixes, [slot] * len(prefixes))
        c, p = grid.configs_to_device(cfgs, pool)
        m, e, s = grid.mask(c, p, len(prefixes))
        torch.cuda.synchronize()
        gm, ge, gs = m.cpu().numpy().view(np.uint32), e.cpu().numpy(), s.cpu().numpy()
        o = oracle_mod.Oracle(rg.text(), drop, rg.lexicon, vocab, specials, eos_id)
        for r, w in enumerate(prefixes):
            ow, oe = o.mask(w, mode=1)
            if not np.array_equal(gm[r], ow) or int(ge[r]) != int(oe):
                diff = np.nonzero(gm[r] != ow)[0]
                toks = [int(k) * 32 + b for k in diff[:4] for b in range(32) if ((int(gm[r][k]) ^ int(ow[k])) >> b) & 1]
                raise AssertionError(f"seed {rg.seed} prefix {w!r}: eos gpu={ge[r]} oracle={oe}, "
                                     f"differing tokens {[(t, vocab[t]) for t in toks[:6]]}")
        assert (gs == 0).all(), (rg.seed, gs)
        n_done += 1


def test_overlay_handoff_to_slow_path(G, oracle_mod):
    """Tokens that shift many terminals (runs of '(' at a boolean position,
    '(' and ')' mixes) outgrow a walk lane's LDS stack area and are finished by
    the slow path; the mask must still equal the oracle's and no row may report
    an overflow."""
    from workloads import grammar_text
    base = make_workload(3, rows=1)
    vocab = [bytes([b]) for b in range(256)]
    vocab += [b"(" * k for k in range(2, 61)] + [b"( " * k for k in range(2, 30)]
    vocab += [b"((a=1)" * k for k in range(1, 9)] + [b")" * k for k in range(2, 20)]
    vocab += [b" (((((((((( 1", b"((((((((((((((((((((((((((((((((((((((((1", b""]
    eos = len(vocab) - 1
    lex = base.lexicons[0]
    g = G.Grid(grammar_text("sql_dml"), base.drop, vocab, [eos], eos)
    slot = g.add_lexicon(lex)
    g.to_device("cuda")
    t, c = base.meta["schema"].tables[0], base.meta["schema"].columns[0][0]
    prefixes = [f"select {c} from {t} where ".encode(), f"select {c} from {t} where ((".encode(),
                f"select {c} from {t} where {c} in (select {c} from {t} where ((((".encode(),
                b"select 1 + ", b"select ("]
    cfgs, pool = g.configs(prefixes, [slot] * len(prefixes))
    cd, pd = g.configs_to_device(cfgs, pool)
    m, e, s = g.mask(cd, pd, len(prefixes))
    torch.cuda.synchronize()
    o = oracle_mod.Oracle(grammar_text("sql_dml"), base.drop, lex, vocab, [eos], eos)
    for i, w in enumerate(prefixes):
        want, want_eos = o.mask(w, mode=1)
        got = m[i].cpu().numpy().view(np.uint32)
        assert np.array_equal(got, want), (w, [vocab[t] for t in range(len(vocab))
                                               if ((int(got[t >> 5]) ^ int(want[t >> 5])) >> (t & 31)) & 1])
        assert int(e[i]) == want_eos
    assert (s.cpu().numpy() == 0).all(), s.cpu().tolist()
    bits = np.unpackbits(m[0].cpu().numpy().view(np.uint8), bitorder="little")
    assert bits[vocab.index(b"(" * 60)] == 1    # a 60-deep run is viable and came back exact


def test_phases_one_call_each_equal_the_whole_call(G):
    """The benchmark's phase pass: prologue, stream, residue and finalize in
    four grid_mask_phases calls give the same masks, EOS flags and status as
    one grid_mask call (workload 3, B = 32), and a second whole call on the
    same workspace gives them again."""
    wl = make_workload(3, rows=32)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    B = len(wl.prefixes)
    cfgs, pool = grid.configs(wl.prefixes, [slot_map[s] for s in wl.slots])
    c, p = grid.configs_to_device(cfgs, pool)
    ws = grid.new_workspace(B, "cuda")
    stream = torch.cuda.current_stream()
    outs = []
    for split in (False, True, False):
        m = torch.empty((B, grid.W), dtype=torch.int32, device="cuda")
        e = torch.empty(B, dtype=torch.uint8, device="cuda")
        s = torch.empty(B, dtype=torch.int32, device="cuda")
        if split:
            for ph in (G.grid.PHASE_PROLOGUE, G.grid.PHASE_WALK, G.grid.PHASE_RESIDUE, G.grid.PHASE_FINALIZE):
                grid.mask(c, p, B, m, e, s, ws, stream, phases=ph)
        else:
            grid.mask(c, p, B, m, e, s, ws, stream)
        torch.cuda.synchronize()
        outs.append((m.cpu().numpy(), e.cpu().numpy(), s.cpu().numpy()))
    for m, e, s in outs[1:]:
        assert np.array_equal(m, outs[0][0]) and np.array_equal(e, outs[0][1]) and np.array_equal(s, outs[0][2])
    assert (outs[0][2] == 0).all()
