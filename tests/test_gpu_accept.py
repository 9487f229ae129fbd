"""grid_accept (device incremental advance, section 6.1 step 7) on the GPU,
anchored to the oracle.

* Decode loops: every row takes a token its exact mask allows, advanced on the
  device with the configurations and stacks the previous step wrote; after
  every step the GPU mask of the advanced configurations equals the oracle's
  mask of the extended prefix w . t word for word (Definition 4), and the
  configuration equals the host advance over the whole prefix.
* Refused tokens, the end-of-sequence token and bad configurations: the
  outputs are the next step's inputs whatever the status, so they are fed
  back into grid_mask and compared with the oracle again.
* The model-free walk arm (section 8.6): 32 rows sample tokens from their GPU
  masks until they choose the end-of-sequence token or 200 steps pass; no
  mask along the way is empty (Proposition 8), every finished output is a
  sentence of the language by the oracle, every unfinished one a viable
  prefix, and the masks are compared with the oracle every 25 steps.
"""

import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import make_workload  # noqa: E402

pytestmark = pytest.mark.gpu

CAP = 1024


def log(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    pkg.lib()
    return pkg


def _host_check(G, grid, prefixes, slots, cfg_out, pool_out, rows, cap=CAP):
    cfgs = cfg_out.cpu().numpy().view(G.CONFIG_DTYPE)
    pool = pool_out.cpu().numpy().view(np.uint16)
    for r in rows:
        want, stack = grid.config(prefixes[r], slots[r])
        got = cfgs[r]
        for f in ("q", "lexnode", "flags", "rem_len", "slot"):
            assert int(got[f]) == int(want[f]), (r, f, prefixes[r][-40:], int(got[f]), int(want[f]))
        assert bytes(got["rem_head"]) == bytes(want["rem_head"]), (r, prefixes[r][-40:])
        off, d = int(got["stk_off"]), int(got["stk_depth"])
        assert off == r * cap and d == len(stack), (r, d, len(stack))
        assert np.array_equal(pool[off:off + d], stack), (r, prefixes[r][-40:])


def _oracle_check(o, wl, prefixes, m, e, s, rows, label):
    """GPU mask rows against the oracle's masks of the same prefixes."""
    got = m.cpu().numpy().view(np.uint32)
    ge = e.cpu().numpy()
    gs = s.cpu().numpy()
    for r in rows:
        want, want_eos = o.mask(prefixes[r], mode=1)
        assert np.array_equal(got[r], want), (label, r, prefixes[r][-60:])
        assert int(ge[r]) == want_eos, (label, r)
        assert gs[r] == 0, (label, r, gs[r])


def _bits(m, V):
    return np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :V]


@pytest.mark.parametrize("k", [2, 3])
def test_accept_decode_loop_matches_oracle_and_host_advance(G, oracle_mod, k):
    wl = make_workload(k, rows=16 if k == 2 else 32)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    o = oracle_mod.from_workload(wl)
    B = len(wl.prefixes)
    slots = [slot_map[s] for s in wl.slots]
    rng = np.random.default_rng(4000 + k)
    prefixes = list(wl.prefixes)
    cfgs, pool = grid.configs(prefixes, slots)
    c, p = grid.configs_to_device(cfgs, pool)
    for step in range(6):
        m, e, s = grid.mask(c, p, B)
        torch.cuda.synchronize()
        bits = _bits(m, wl.V)
        toks = np.zeros(B, np.int32)
        for r in range(B):
            allowed = np.flatnonzero(bits[r])
            allowed = allowed[allowed != wl.eos_id]
            toks[r] = rng.choice(allowed) if len(allowed) else (wl.eos_id if wl.eos_id >= 0 else 0)
        t = torch.from_numpy(toks).to("cuda")
        c2, p2, st = grid.accept(c, p, t, B, CAP)
        torch.cuda.synchronize()
        st = st.cpu().numpy()
        ok = [r for r in range(B) if toks[r] != wl.eos_id]
        assert (st[ok] == G.ROW_OK).all(), (step, st.tolist())
        for r in ok:
            prefixes[r] = prefixes[r] + wl.vocab[toks[r]]
        _host_check(G, grid, prefixes, slots, c2, p2, ok)
        c, p = c2, p2.view(torch.int16)
        # the mask of every advanced configuration is the oracle's mask of w . t
        m, e, s = grid.mask(c, p, B)
        torch.cuda.synchronize()
        _oracle_check(o, wl, prefixes, m, e, s, ok, f"workload {k} step {step}")
        log(f"workload {k} step {step}: {len(ok)} rows advanced; masks equal the oracle's, "
            f"configurations equal the host advance")
    # blocked tokens are refused; the row keeps its configuration, and the
    # outputs fed back give the same masks as before (the oracle's)
    m, e, s = grid.mask(c, p, B)
    torch.cuda.synchronize()
    bits = _bits(m, wl.V)
    toks = np.zeros(B, np.int32)
    for r in range(B):
        blocked = np.flatnonzero(bits[r] == 0)
        blocked = blocked[blocked != wl.eos_id]
        toks[r] = rng.choice(blocked)
    c3, p3, st = grid.accept(c, p, torch.from_numpy(toks).to("cuda"), B, CAP)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == G.ROW_NOT_VIABLE).all()
    _host_check(G, grid, prefixes, slots, c3, p3, range(B))
    m3, e3, s3 = grid.mask(c3, p3.view(torch.int16), B)
    torch.cuda.synchronize()
    assert np.array_equal(m3.cpu().numpy(), m.cpu().numpy())
    _oracle_check(o, wl, prefixes, m3, e3, s3, range(B), f"workload {k} refused")
    # the end-of-sequence token finishes exactly the rows whose mask allows
    # it; their outputs still hold their configurations
    if wl.eos_id >= 0:
        eos_tok = torch.full((B,), wl.eos_id, dtype=torch.int32, device="cuda")
        c4, p4, st = grid.accept(c, p, eos_tok, B, CAP)
        torch.cuda.synchronize()
        want = np.where(e.cpu().numpy() != 0, G.ROW_FINISHED, G.ROW_NOT_VIABLE)
        assert np.array_equal(st.cpu().numpy(), want)
        _host_check(G, grid, prefixes, slots, c4, p4, range(B))


def test_accept_edge_cases(G, oracle_mod):
    """Empty prefixes, a sentence end, a configuration out of range, a stack
    capacity too small."""
    wl = make_workload(3, rows=1)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    vocab = {t: i for i, t in enumerate(wl.vocab)}
    prefixes = [b"", b"", b"select 1", b"select 1"]
    toks = [vocab[b"s"], vocab[b" "], vocab[b";"], vocab[b"s"]]
    slots = [slot_map[0]] * len(prefixes)
    cfgs, pool = grid.configs(prefixes, slots)
    bad = cfgs.copy()
    c, p = grid.configs_to_device(cfgs, pool)
    c2, p2, st = grid.accept(c, p, torch.tensor(toks, dtype=torch.int32, device="cuda"), len(prefixes), CAP)
    torch.cuda.synchronize()
    st = st.cpu().numpy()
    assert st[0] == G.ROW_OK and st[2] == G.ROW_OK, st
    ext = [prefixes[i] + wl.vocab[toks[i]] for i in range(len(prefixes))]
    # b" " from the empty prefix and "select 1" + "s" are (not) viable as the host says
    for i in (1, 3):
        try:
            grid.config(ext[i], slots[i])
            viable = True
        except G.GridError:
            viable = False
        assert (st[i] == G.ROW_OK) == viable, (i, st[i], viable)
    _host_check(G, grid, ext, slots, c2, p2, [0, 2])
    bad["q"][0] = 60000
    cb, pb = grid.configs_to_device(bad, pool)
    _, _, st = grid.accept(cb, pb, torch.tensor(toks, dtype=torch.int32, device="cuda"), len(prefixes), CAP)
    c5, p5, st2 = grid.accept(c, p, torch.tensor(toks, dtype=torch.int32, device="cuda"), len(prefixes), 2)
    torch.cuda.synchronize()
    assert st.cpu().numpy()[0] == G.ROW_BAD_CONFIG
    st2 = st2.cpu().numpy()
    assert st2[2] in (G.ROW_OVERFLOW, G.ROW_BAD_CONFIG)
    # a stack that does not fit the capacity leaves depth 0: fed back, the
    # mask reports a bad configuration
    depths = c5.cpu().numpy().view(G.CONFIG_DTYPE)["stk_depth"]
    for r in range(len(prefixes)):
        if len(grid.config(prefixes[r], slots[r])[1]) > 2:
            assert st2[r] == G.ROW_BAD_CONFIG and depths[r] == 0, (r, st2[r], depths[r])
    _, _, sm = grid.mask(c5, p5.view(torch.int16), len(prefixes))
    torch.cuda.synchronize()
    assert all((sm.cpu().numpy()[r] == G.ROW_BAD_CONFIG) == (depths[r] == 0) for r in range(len(prefixes)))


def test_accept_rejects_out_of_range_lexnode_and_stack_entry(G, oracle_mod):
    """A lexicon node beyond its slot's trie and a stack entry that is no LR
    state are reported as bad configurations (nothing is read through them);
    the other rows of the batch advance normally, and every output fed back
    into grid_mask gives the oracle's mask or the bad-configuration status."""
    wl = make_workload(3, rows=1)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    o = oracle_mod.from_workload(wl)
    vocab = {t: i for i, t in enumerate(wl.vocab)}
    s0 = slot_map[0]
    t0 = wl.meta["schema"].tables[0]
    prefixes = [f"select * from {t0[:2]}".encode(), b"select 1", b"select (1", f"select * from {t0[:2]}".encode()]
    toks = [vocab[bytes([t0[2].encode()[0]])], vocab[b" "], vocab[b")"], vocab[bytes([t0[2].encode()[0]])]]
    cfgs, pool = grid.configs(prefixes, [s0] * len(prefixes))
    assert cfgs["lexnode"][0] != 0xFFFFFFFF
    bad = cfgs.copy()
    bad["lexnode"][0] = 0x7FFFFFF0                    # beyond the slot's node count
    pool = pool.copy()
    off2, d2 = int(cfgs["stk_off"][2]), int(cfgs["stk_depth"][2])
    pool[off2 + d2 // 2] = 0xFFF0                     # no LR state has this number
    c, p = grid.configs_to_device(bad, pool)
    c2, p2, st = grid.accept(c, p, torch.tensor(toks, dtype=torch.int32, device="cuda"), len(prefixes), CAP)
    torch.cuda.synchronize()
    st = st.cpu().numpy()
    assert st[0] == G.ROW_BAD_CONFIG and st[2] == G.ROW_BAD_CONFIG, st
    assert st[1] == G.ROW_OK and st[3] == G.ROW_OK, st
    m, e, s = grid.mask(c2, p2.view(torch.int16), len(prefixes))
    torch.cuda.synchronize()
    s = s.cpu().numpy()
    assert s[0] == G.ROW_BAD_CONFIG and s[2] == G.ROW_BAD_CONFIG, s
    ext = [prefixes[i] + wl.vocab[toks[i]] for i in range(len(prefixes))]
    _oracle_check(o, wl, ext, m, e, torch.from_numpy(s), [1, 3], "good rows beside bad ones")


@pytest.mark.parametrize("k", [2, 3])
def test_walk_arm_sampled_until_end_of_sequence(G, oracle_mod, k):
    wl = make_workload(k, rows=32)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    o = oracle_mod.from_workload(wl)
    B = len(wl.prefixes)
    slots = [slot_map[s] for s in wl.slots]
    cap = 4096
    rng = np.random.default_rng(8600 + k)
    ids = {sp: i for i, sp in enumerate(wl.vocab)}
    # after 50 steps the walk leans toward spellings that close what is open
    # (strings, comments, parentheses, expressions, the statement); this
    # shapes how often a walk ends, not what the checks accept
    closers = [ids[x] for x in (b")", b";", b"'", b" ", b"\n", b" end", b" 1") if x in ids]
    prefixes = list(wl.prefixes)
    cfgs, pool = grid.configs(prefixes, slots)
    c, p = grid.configs_to_device(cfgs, pool)
    finished = np.zeros(B, bool)
    for step in range(200):
        m, e, s = grid.mask(c, p, B)
        torch.cuda.synchronize()
        bits = _bits(m, wl.V)
        ge = e.cpu().numpy()
        gs = s.cpu().numpy()
        live = [r for r in range(B) if not finished[r]]
        assert (gs[live] == 0).all(), (step, gs.tolist())
        for r in live:   # no mask is empty at a viable configuration
            assert bits[r].any() or ge[r], (step, r, prefixes[r][-60:])
        if step % 25 == 0:
            _oracle_check(o, wl, prefixes, m, e, s, live, f"walk {k} step {step}")
        toks = np.full(B, wl.eos_id, np.int32)
        for r in live:
            allowed = np.flatnonzero(bits[r])
            allowed = allowed[allowed != wl.eos_id]
            if ge[r] and (len(allowed) == 0 or rng.random() < (0.3 if step < 50 else 0.9)):
                continue  # the end-of-sequence token
            tok = int(rng.choice(allowed))
            if step >= 50 and rng.random() < 0.7:
                cand = [x for x in closers if bits[r][x]]
                if cand:
                    tok = int(rng.choice(cand))
            toks[r] = tok
        c2, p2, st = grid.accept(c, p, torch.from_numpy(toks).to("cuda"), B, cap)
        torch.cuda.synchronize()
        st = st.cpu().numpy()
        for r in live:
            if toks[r] == wl.eos_id:
                assert st[r] == G.ROW_FINISHED, (step, r, st[r])
                finished[r] = True
            else:
                assert st[r] == G.ROW_OK, (step, r, st[r])
                prefixes[r] = prefixes[r] + wl.vocab[toks[r]]
        c, p = c2, p2.view(torch.int16)
        if finished.all():
            break
    n_fin = int(finished.sum())
    for r in range(B):
        if finished[r]:
            assert o.member(prefixes[r]), (r, prefixes[r][-80:])
        else:
            assert o.viable(prefixes[r]), (r, prefixes[r][-80:])
    log(f"walk arm, workload {k}: {n_fin} of {B} rows ended with the end-of-sequence token "
        f"(all members of L by the oracle), the rest viable after {step + 1} steps; no empty mask")
    assert n_fin >= 4


def test_accept_deep_stacks_leave_the_lds_area(G):
    """Stacks deeper than the kernel keeps in LDS (8192 entries) with a larger
    capacity: a row that starts above that depth, one that crosses it during
    the decode loop and a shallow one, advanced by "((" three times, equal the
    host advance at every step."""
    wl = make_workload(3, rows=1)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    vocab = {t: i for i, t in enumerate(wl.vocab)}
    cap = 16384
    prefixes = [b"select " + b"(" * 8186, b"select " + b"(" * 9000, b"select ("]
    slots = [slot_map[0]] * len(prefixes)
    cfgs, pool = grid.configs(prefixes, slots)
    c, p = grid.configs_to_device(cfgs, pool)
    tok = vocab[b"(("]
    t = torch.full((len(prefixes),), tok, dtype=torch.int32, device="cuda")
    for step in range(3):
        c2, p2, st = grid.accept(c, p, t, len(prefixes), cap)
        torch.cuda.synchronize()
        assert (st.cpu().numpy() == G.ROW_OK).all(), (step, st.cpu().numpy().tolist())
        prefixes = [x + b"((" for x in prefixes]
        _host_check(G, grid, prefixes, slots, c2, p2, range(len(prefixes)), cap)
        depths = c2.cpu().numpy().view(G.CONFIG_DTYPE)["stk_depth"].tolist()
        log(f"deep stacks step {step}: depths {depths} equal to the host advance")
        c, p = c2, p2.view(torch.int16)
    # a refused token on the deep rows (the global route rewrites the output
    # copy as it goes) leaves the input stack in the output area
    bad_tok = torch.full((len(prefixes),), vocab[b";"], dtype=torch.int32, device="cuda")
    c3, p3, st = grid.accept(c, p, bad_tok, len(prefixes), cap)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == G.ROW_NOT_VIABLE).all()
    _host_check(G, grid, prefixes, slots, c3, p3, range(len(prefixes)), cap)
