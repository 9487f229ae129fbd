"""Random-grammar campaign on the GPU: N random LALR(1) grammars (seeds from
START on; one in three with 8..14 nonterminals, one in four under a role
projection that drops one or two labelled alternatives), each with its own vocabulary
of 2,500 tokens of up to 12 bytes (half of them strings of several lexemes,
so byte walks emit several terminals) and 8, 32 or 48 sampled prefixes in one
batch; every mask, end-of-sequence byte and row status is compared with the
oracle's (checkpoint mode).  With "decode", each batch then runs 8 decode
steps: a token sampled from every row's GPU mask is accepted in place
(grid_accept_inplace on per-row stack regions), the configuration and stack
must equal the host advance of the extended prefix, and the next mask the
oracle's.  Stops at the first difference and prints it.

    python tests/random_campaign.py START N [decode]

Not collected by pytest (a longer run than the test suite's random-grammar
cases); it uses the oracle, so it lives with the tests.
"""

import random
import sys
import time
from pathlib import Path

import numpy as np

sys.path.insert(0, str(Path(__file__).resolve().parent.parent))


def vocabulary(rg, r):
    alpha = rg.alphabet()
    words = sorted({w for ws in (rg.lexicon or {}).values() for w in ws})
    vocab = [bytes([b]) for b in range(0x20, 0x7F)]
    seen = set(vocab)
    for w in words:
        for t in (w.encode(), (" " + w).encode()):
            if t not in seen:
                seen.add(t)
                vocab.append(t)
    lexemes = list(rg.literal.values()) + words + ["12", "7", "ab", "x1"]
    while len(vocab) < 2500:
        if r.random() < 0.5:  # several lexemes in one token
            s = "".join(r.choice(lexemes) + (" " if r.random() < 0.4 else "") for _ in range(r.randint(2, 5)))[:12]
        else:
            s = "".join(r.choice(alpha) for _ in range(r.randint(2, 12)))
        t = s.encode()
        if t not in seen:
            seen.add(t)
            vocab.append(t)
    eos = len(vocab)
    vocab.append(b"")
    return vocab, eos


def compare(vocab, rg, gm, ge, gs, o, prefixes, B, what):
    for i, w in enumerate(prefixes):
        ow, oe = o.mask(w, mode=1)
        if not np.array_equal(gm[i], ow) or int(ge[i]) != int(oe) or gs[i] != 0:
            diff = np.nonzero(gm[i] != ow)[0]
            toks = [int(k) * 32 + b for k in diff[:6] for b in range(32) if ((int(gm[i][k]) ^ int(ow[k])) >> b) & 1]
            print(f"difference ({what}): seed {rg.seed} B {B} row {i} prefix {w!r} status {gs[i]} "
                  f"eos {ge[i]}/{oe} tokens {[(t, vocab[t]) for t in toks[:8]]}", flush=True)
            print(rg.text(), rg.lexicon, flush=True)
            return False
    return True



def decode(G, grid, slot, vocab, eos, rg, o, prefixes, rng, steps=8, cap=512):
    """Decode steps with the in-place advance; False at the first difference."""
    import torch
    B = len(prefixes)
    prefixes = list(prefixes)
    cfgs, pool = grid.configs(prefixes, [slot] * B)
    region = np.zeros(B * cap, dtype=np.uint16)
    for b in range(B):
        off, d = int(cfgs["stk_off"][b]), int(cfgs["stk_depth"][b])
        region[b * cap:b * cap + d] = pool[off:off + d]
        cfgs["stk_off"][b] = b * cap
    c, p = grid.configs_to_device(cfgs, region)
    for step in range(steps):
        m, e, st = grid.mask(c, p, B)
        torch.cuda.synchronize()
        bits = np.unpackbits(m.cpu().numpy().view(np.uint8), axis=1, bitorder="little")[:, :len(vocab)]
        toks = np.zeros(B, np.int32)
        for r in range(B):
            allowed = np.flatnonzero(bits[r])
            rest = allowed[allowed != eos]
            toks[r] = rng.choice(rest) if len(rest) else eos
        acc = grid.accept_inplace(c, p, torch.from_numpy(toks).cuda(), B, cap).cpu().numpy()
        for r in range(B):
            want_status = G.ROW_FINISHED if toks[r] == eos else G.ROW_OK
            if acc[r] != want_status:
                print(f"difference (accept status): seed {rg.seed} row {r} step {step} {acc[r]}", flush=True)
                return False
            if toks[r] != eos:
                prefixes[r] += vocab[toks[r]]
        got = c.cpu().numpy().view(G.CONFIG_DTYPE)
        pool_now = p.cpu().numpy().view(np.uint16)
        for r in range(B):
            want, stack = grid.config(prefixes[r], slot)
            off, d = int(got[r]["stk_off"]), int(got[r]["stk_depth"])
            same = all(int(got[r][f]) == int(want[f]) for f in ("q", "lexnode", "flags", "rem_len", "slot"))
            same = same and bytes(got[r]["rem_head"]) == bytes(want["rem_head"])
            same = same and d == len(stack) and np.array_equal(pool_now[off:off + d], stack)
            if not same:
                print(f"difference (advance): seed {rg.seed} row {r} step {step} prefix {prefixes[r]!r}", flush=True)
                return False
        m, e, st = grid.mask(c, p, B)
        torch.cuda.synchronize()
        if not compare(vocab, rg, m.cpu().numpy().view(np.uint32), e.cpu().numpy(), st.cpu().numpy(), o, prefixes,
                       B, f"decode step {step}"):
            return False
    return True


def main(start, n_want, with_decode=False):
    import torch
    import oracle
    import paper_2607_11951_amd as G
    from workloads.randgram import RandomGrammar
    t0 = time.time()
    done = tried = rows = 0
    seed = start
    while done < n_want:
        rg = RandomGrammar(seed, n_nt=None if seed % 3 else 8 + seed % 7)
        seed += 1
        tried += 1
        r = random.Random(seed * 7)
        vocab, eos = vocabulary(rg, r)
        drop = rg.random_drop(r, r.randint(1, 2)) if seed % 4 == 0 else []
        try:
            grid = G.Grid(rg.text(), drop, vocab, [eos], eos)
        except G.GridError as e:
            assert "GRID_E_LALR_CONFLICT" in str(e) or "GRID_E_EMPTY_LANGUAGE" in str(e), str(e)
            continue
        slot = grid.add_lexicon(rg.lexicon) if rg.lexicon else 0
        grid.to_device("cuda")
        B = r.choice([8, 32, 48])
        rr = random.Random(seed)
        prefixes = []
        while len(prefixes) < B:
            s = rg.sentence(rr, max_depth=10, max_len=120, drop=drop)
            prefixes.append(s[:rr.randint(0, len(s))] if rr.random() < 0.9 else s)
        cfgs, pool = grid.configs(prefixes, [slot] * B)
        c, p = grid.configs_to_device(cfgs, pool)
        m, e, st = grid.mask(c, p, B)
        torch.cuda.synchronize()
        gm, ge, gs = m.cpu().numpy().view(np.uint32), e.cpu().numpy(), st.cpu().numpy()
        o = oracle.Oracle(rg.text(), drop, rg.lexicon, vocab, [eos], eos)
        if not compare(vocab, rg, gm, ge, gs, o, prefixes, B, "mask"):
            return 1
        if with_decode and not decode(G, grid, slot, vocab, eos, rg, o, prefixes, np.random.default_rng(seed)):
            return 1
        rows += B
        done += 1
        if done % 25 == 0:
            print(f"{done} grammars ({tried} tried), {rows} rows, {time.time() - t0:.0f} s, last seed {rg.seed}",
                  flush=True)
    print(f"all equal: {done} grammars, {rows} rows, {time.time() - t0:.0f} s", flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main(int(sys.argv[1]), int(sys.argv[2]), len(sys.argv) > 3 and sys.argv[3] == "decode"))
