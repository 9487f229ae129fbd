"""grid_mask_noalloc (the mask entry point that allocates nothing: its
workspace is the library's static device scratch array) through the C ABI,
against grid_mask with a caller workspace, bit for bit: two calls in a row on
the benchmark's workload (B = 32, V = 151,936), the second with a smaller
batch of other rows, so the second call runs over what the first left in the
array; then a batch too large for the array is refused before any launch."""

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from workloads import make_workload  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def G():
    import paper_2607_11951_amd as pkg
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    pkg.lib()
    return pkg


def _both(G, grid, wl, slots, rows):
    cfgs, pool = grid.configs([wl.prefixes[j] for j in rows], [slots[wl.slots[j]] for j in rows])
    c, p = grid.configs_to_device(cfgs, pool)
    B = len(rows)
    ref = grid.mask(c, p, B)
    out = (torch.full((B, grid.W), -1, dtype=torch.int32, device="cuda"),
           torch.full((B,), 7, dtype=torch.uint8, device="cuda"),
           torch.full((B,), -1, dtype=torch.int32, device="cuda"))
    got = G.mask_noalloc(grid, c, p, B, *out)
    torch.cuda.synchronize()
    return [x.cpu().numpy() for x in ref], [x.cpu().numpy() for x in got]


def test_noalloc_equals_grid_mask_two_calls(G):
    wl = make_workload(3, n_batches=2)
    grid, slots = G.from_workload(wl)
    grid.to_device("cuda")
    lib = G.lib()
    assert grid.workspace_bytes(32) <= lib.grid_mask_noalloc_max_bytes()
    for rows in (list(range(32)), list(range(40, 48))):
        ref, got = _both(G, grid, wl, slots, rows)
        for a, b, what in zip(ref, got, ("mask", "eos", "status")):
            assert np.array_equal(a, b), (len(rows), what)
        assert (got[2] == 0).all()
    # a batch whose workspace exceeds the static array is refused up front
    big = 1
    while grid.workspace_bytes(big) <= lib.grid_mask_noalloc_max_bytes():
        big *= 2
    cfgs, pool = grid.configs([wl.prefixes[0]] * big, [slots[wl.slots[0]]] * big)
    c, p = grid.configs_to_device(cfgs, pool)
    out = (torch.empty((big, grid.W), dtype=torch.int32, device="cuda"),
           torch.empty(big, dtype=torch.uint8, device="cuda"), torch.empty(big, dtype=torch.int32, device="cuda"))
    with pytest.raises(G.GridError) as ei:
        G.mask_noalloc(grid, c, p, big, *out)
    assert ei.value.code == -11


def test_noalloc_small_grammar_after_large(G):
    """A different grammar on the same array right after: workload 2's rows."""
    wl = make_workload(2, rows=20)
    grid, slots = G.from_workload(wl)
    grid.to_device("cuda")
    ref, got = _both(G, grid, wl, slots, list(range(20)))
    for a, b, what in zip(ref, got, ("mask", "eos", "status")):
        assert np.array_equal(a, b), what
