"""The allocation-free page-table build (colour_alloc_pagetable_noalloc)
through the C ABI, against the allocating build (colour_alloc_pagetable):
the same table and count bit for bit on two calls in a row, the second with
a smaller pool and fewer pages (the fixed scratch keeps the first call's
contents), a shortfall (reported through the count, no error) and the size
limit of the fixed scratch."""
import sys

import numpy as np
import pytest

import synth
import paper_2407_13996_amd as sg

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")
DEV = "cuda:0"


def say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(scope="module")
def ctx():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    c = sg.Context(0)
    yield c
    c.close()


def both(ctx, masks, origin, shift, pool, S, n):
    ref = torch.full((max(n, 1),), -1, dtype=torch.int32, device=DEV)
    try:
        found = sg.colour_alloc_pagetable(ctx, masks, origin, shift, pool, S, n, ref)
    except sg.SgdrcError as e:
        assert e.code == sg.ENOMEM
        found = e.n_found
    got = torch.full((max(n, 1),), -7, dtype=torch.int32, device=DEV)
    got_n = torch.full((1,), -1, dtype=torch.int64, device=DEV)
    sg.colour_alloc_pagetable_noalloc(ctx, masks, origin, shift, pool, S, n, got, got_n)
    torch.cuda.synchronize()
    k = min(found, n)
    return found, int(got_n.item()), ref[:k].cpu().numpy(), got[:k].cpu().numpy(), got[k:]


def test_noalloc_pagetable_matches_the_allocating_build(ctx):
    masks = synth.xor_masks(6, seed=1, min_bit=16)
    # the streaming triad's pool at 8 of 64 colours (three 1 GiB arrays), then a smaller pool and table
    for origin, shift, pool, S, n in [(1 << 36, 16, 393216, range(8), 3 * 16384),
                                      (1 << 40, 16, 50000, range(16, 40), 3000)]:
        say(f"noalloc page table: pool {pool} pages of {1 << (shift - 10)} KiB, |S| {len(S)}, n {n}")
        found, got_found, ref, got, rest = both(ctx, masks, origin, shift, pool, S, n)
        assert got_found == found >= n
        assert (got.view(np.uint32) == ref.view(np.uint32)).all()
        assert bool((rest == -7).all())
    # a shortfall is reported through the count: every qualifying page written
    found, got_found, ref, got, rest = both(ctx, masks, 0, 16, 2000, [5], 1000)
    assert got_found == found < 1000
    assert (got.view(np.uint32) == ref.view(np.uint32)).all()
    assert bool((rest == -7).all())


def test_noalloc_pagetable_limits(ctx):
    masks = synth.xor_masks(6, seed=1, min_bit=16)
    pt = torch.zeros(16, dtype=torch.int32, device=DEV)
    n = torch.zeros(1, dtype=torch.int64, device=DEV)
    with pytest.raises(sg.SgdrcError) as e:
        sg.colour_alloc_pagetable_noalloc(ctx, masks, 0, 16, (1 << 26) + 1, [0], 16, pt, n)
    assert e.value.code == sg.EINVAL and str(1 << 26) in str(e.value)
    with pytest.raises(sg.SgdrcError) as e:
        sg.colour_alloc_pagetable_noalloc(ctx, masks, 0, 16, 1024, [0], 16, pt, None)
    assert e.value.code == sg.EINVAL
    # the largest pool the fixed scratch serves
    found, got_found, ref, got, rest = both(ctx, masks, 1 << 38, 10, 1 << 26, [0], 1 << 16)
    assert got_found == found and (got.view(np.uint32) == ref.view(np.uint32)).all()
