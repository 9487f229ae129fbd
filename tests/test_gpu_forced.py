"""Jump-forward forced spans (section 6.1 step 6) on the GPU through the C
ABI (grid_forced_span), checked by the oracle.

The expected span of a prefix is written out from the oracle's masks: while
the mask (with the end-of-sequence bit when the prefix is a sentence) has
exactly one bit, that token is appended, and the end-of-sequence token ends
the span; max_len bounds it.  For every row the device span, its length, the
mask of the final configuration, the final configuration and stack (against
the host advance of the extended prefix) and the kept rolling hashes are
compared.

* A CRUD grammar (analyst role) with a coarse vocabulary and a one-table
  lexicon, whose prefixes have forced spans of 0 to 5 tokens, the
  end-of-sequence token and the max_len bound included.
* Rows of the DML workload (151,936 tokens), where forced steps are rare:
  most spans are empty and the final mask is the plain mask.
"""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import grammar_text, make_workload  # noqa: E402

pytestmark = pytest.mark.gpu

CAP = 1024


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    pkg.lib()
    return pkg


def _regions(grid, prefixes, slots, cap=CAP):
    cfgs, pool = grid.configs(prefixes, slots)
    region = np.zeros(len(prefixes) * cap, dtype=np.uint16)
    for b in range(len(prefixes)):
        off, d = int(cfgs["stk_off"][b]), int(cfgs["stk_depth"][b])
        region[b * cap:b * cap + d] = pool[off:off + d]
        cfgs["stk_off"][b] = b * cap
    return cfgs, region


def _bits(words, V):
    return np.flatnonzero(np.unpackbits(np.asarray(words, np.uint32).view(np.uint8), bitorder="little")[:V])


def _oracle_span(o, vocab, eos_id, w, max_len):
    span = []
    while len(span) < max_len:
        words, _ = o.mask(w, mode=1)
        allowed = _bits(words, len(vocab))
        if len(allowed) != 1:
            break
        t = int(allowed[0])
        span.append(t)
        if t == eos_id:
            break
        w += vocab[t]
    return span, w


def _check(G, grid, o, vocab, eos_id, prefixes, slots, max_len):
    B = len(prefixes)
    cfgs, region = _regions(grid, prefixes, slots)
    c, p = grid.configs_to_device(cfgs, region)
    h = grid.stack_hash(c, p, B)
    span, n, m, e, s = grid.forced_span(c, p, B, CAP, max_len, stack_hash=h)
    torch.cuda.synchronize()
    span, n, m = span.cpu().numpy(), n.cpu().numpy(), m.cpu().numpy().view(np.uint32)
    e, s = e.cpu().numpy(), s.cpu().numpy()
    got = c.cpu().numpy().view(G.CONFIG_DTYPE)
    pool = p.cpu().numpy().view(np.uint16)
    hashes = h.cpu().numpy().view(np.uint64)
    lengths = []
    for r, w in enumerate(prefixes):
        want, end = _oracle_span(o, vocab, eos_id, w, max_len)
        assert int(n[r]) == len(want), (r, w, span[r].tolist(), want)
        assert span[r, :len(want)].tolist() == want and (span[r, len(want):] == -1).all(), (r, w)
        assert s[r] == G.ROW_OK
        wm, we = o.mask(end, mode=1)
        assert np.array_equal(m[r], wm) and int(e[r]) == we, (r, end)
        cfg, stack = grid.config(end, slots[r])
        for f in ("q", "lexnode", "flags", "rem_len", "slot"):
            assert int(got[r][f]) == int(cfg[f]), (r, f)
        off, d = int(got[r]["stk_off"]), int(got[r]["stk_depth"])
        assert off == r * CAP and d == len(stack) and np.array_equal(pool[off:off + d], stack), r
        assert np.array_equal(hashes[off:off + d], grid.stack_hash_host(stack)), r
        lengths.append(len(want))
    return lengths


def test_forced_spans_crud(G, oracle_mod):
    vocab = [b"select", b" *", b" from", b" employees", b";", b" where", b" id", b" =", b" 1", b"<eos>"]
    eos = len(vocab) - 1
    lex = {"TABLE_NAME": ["employees"], "COLUMN_NAME": ["id"]}
    drop = ["insert", "update", "delete"]
    grid = G.Grid(grammar_text("crud"), drop, vocab, [eos], eos)
    slot = grid.add_lexicon(lex)
    grid.to_device("cuda")
    o = oracle_mod.Oracle(grammar_text("crud"), drop, lex, vocab, [eos], eos)
    prefixes = [b"", b"select", b"select *", b"select * from employees where", b"select * from employees",
                b"select * from employees where id = 1 and", b"select * from employees;"]
    for max_len in (1, 3, 8):
        lengths = _check(G, grid, o, vocab, eos, prefixes, [slot] * len(prefixes), max_len)
        if max_len == 8:
            assert lengths == [1, 0, 2, 5, 0, 5, 1], lengths   # "select" ... the end-of-sequence token
        else:
            assert max(lengths) == max_len, lengths


def test_forced_spans_dml_rows(G, oracle_mod):
    wl = make_workload(3, rows=12)
    grid, sm = G.from_workload(wl)
    grid.to_device("cuda")
    o = oracle_mod.from_workload(wl)
    lengths = _check(G, grid, o, wl.vocab, wl.eos_id, list(wl.prefixes), [sm[s] for s in wl.slots], 4)
    print(f"DML forced span lengths: {lengths}", flush=True)
