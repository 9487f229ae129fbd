"""grid_accept (device incremental advance, section 6.1 step 7) against the
host advance: a decode loop of several steps in which every row takes a
token its exact mask allows, run on the device with the configurations and
stacks the previous step wrote, must reach the same configuration -- stack,
lexer state, lexicon node, pending bytes -- as the host advance over the
whole extended prefix; tokens the mask blocks are refused and leave the
configuration as it was; the end-of-sequence token finishes exactly the rows
whose mask allows it."""

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


@pytest.mark.parametrize("k", [2, 3])
def test_accept_decode_loop_matches_host_advance(G, k):
    wl = make_workload(k, rows=16 if k == 2 else 32)
    grid, slot_map = G.from_workload(wl)
    grid.to_device("cuda")
    B = len(wl.prefixes)
    slots = [slot_map[s] for s in wl.slots]
    rng = np.random.default_rng(4000 + k)
    prefixes = list(wl.prefixes)
    cfgs, pool = grid.configs(prefixes, slots)
    c, p = grid.configs_to_device(cfgs, pool)
    live = list(range(B))
    for step in range(6):
        m, e, s = grid.mask(c, p, B)
        torch.cuda.synchronize()
        bits = np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
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
        log(f"workload {k} step {step}: {len(ok)} rows advanced and equal to the host advance")
        c, p = c2, p2.view(torch.int16)
    # blocked tokens are refused, the configuration stays
    m, e, s = grid.mask(c, p, B)
    torch.cuda.synchronize()
    bits = np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :wl.V]
    toks = np.zeros(B, np.int32)
    for r in range(B):
        blocked = np.flatnonzero(bits[r] == 0)
        blocked = blocked[blocked != wl.eos_id]
        toks[r] = rng.choice(blocked)
    c3, p3, st = grid.accept(c, p, torch.from_numpy(toks).to("cuda"), B, CAP)
    torch.cuda.synchronize()
    assert (st.cpu().numpy() == G.ROW_NOT_VIABLE).all()
    assert np.array_equal(c3.cpu().numpy(), c.cpu().numpy())
    # the end-of-sequence token finishes exactly the rows whose mask allows it
    if wl.eos_id >= 0:
        eos_tok = torch.full((B,), wl.eos_id, dtype=torch.int32, device="cuda")
        _, _, st = grid.accept(c, p, eos_tok, B, CAP)
        torch.cuda.synchronize()
        want = np.where(e.cpu().numpy() != 0, G.ROW_FINISHED, G.ROW_NOT_VIABLE)
        assert np.array_equal(st.cpu().numpy(), want)


def test_accept_edge_cases(G):
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
    _, _, st2 = grid.accept(c, p, torch.tensor(toks, dtype=torch.int32, device="cuda"), len(prefixes), 2)
    torch.cuda.synchronize()
    assert st.cpu().numpy()[0] == G.ROW_BAD_CONFIG
    assert st2.cpu().numpy()[2] in (G.ROW_OVERFLOW, G.ROW_BAD_CONFIG)


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
