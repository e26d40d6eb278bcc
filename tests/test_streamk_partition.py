"""Host model of the stream-K work partition of the contraction kernel.

The kernel gives logical work-group g the (tile, K-block) iterations
[start(g), start(g+1)), start(g) = floor(g*T/G), walks them as segments
that end at tile boundaries, finds a tile's contributors with owner() and
stores partial tiles in slot 2g (first tile of the range) or 2g+1.  These
checks run the same integer formulas on the CPU over many shapes: every
iteration is computed exactly once, owner() names exactly the work-groups
that hold a segment of the tile, partial slots never collide and stay below
2G, and the XCD renumbering of work-group ids is a permutation.
"""
import itertools

import pytest


def start(g, T, G):
    return (g * T) // G


def owner(i, T, G):
    return ((i + 1) * G + T - 1) // T - 1


def slot(g, t, T, G, nkb):
    return 2 * g if start(g, T, G) // nkb == t else 2 * g + 1


def segments(g, T, G, nkb):
    """The (tile, kbeg, kend) segments work-group g walks, as the kernel does."""
    seg, end = start(g, T, G), start(g + 1, T, G)
    out = []
    while seg < end:
        tile = seg // nkb
        kbeg = seg - tile * nkb
        kend = min(nkb, kbeg + (end - seg))
        out.append((tile, kbeg, kend))
        seg += kend - kbeg
    return out


def logical(b, G, xcds):
    if xcds > 1 and G % xcds == 0:
        return (b % xcds) * (G // xcds) + b // xcds
    return b


CASES = [(tiles, nkb, G) for tiles, nkb, G in itertools.product(
    [1, 2, 3, 7, 52, 196, 785], [1, 2, 5, 18, 72, 144], [1, 8, 24, 256, 512, 768, 1024])
    if G <= tiles * nkb]


@pytest.mark.parametrize("tiles,nkb,G", CASES)
def test_streamk_partition(tiles, nkb, G):
    T = tiles * nkb
    covered = [0] * T
    holders = {}          # tile -> work-groups with a segment in it
    slots = {}
    for g in range(G):
        segs = segments(g, T, G, nkb)
        assert segs, "every work-group has at least one iteration"
        for tile, kbeg, kend in segs:
            assert 0 <= kbeg < kend <= nkb
            for k in range(kbeg, kend):
                covered[tile * nkb + k] += 1
            holders.setdefault(tile, []).append((g, kbeg, kend))
    assert all(c == 1 for c in covered)
    for tile, hs in holders.items():
        lo, hi = owner(tile * nkb, T, G), owner(tile * nkb + nkb - 1, T, G)
        assert [g for g, _, _ in hs] == list(range(lo, hi + 1))
        # contributors in increasing g hold increasing K-blocks: the kernel's
        # summation order g = lo .. hi is the order of the reduction
        assert [k for _, k, _ in hs] == sorted(k for _, k, _ in hs)
        full = len(hs) == 1
        assert full == (hs[0][1] == 0 and hs[0][2] == nkb)
        if not full:
            for g, _, _ in hs:
                s = slot(g, tile, T, G, nkb)
                assert 0 <= s < 2 * G
                assert s not in slots, (g, tile, slots.get(s))
                slots[s] = (g, tile)


@pytest.mark.parametrize("G,xcds", [(8, 8), (512, 8), (768, 8), (24, 8), (7, 8), (256, 1)])
def test_xcd_renumbering_is_a_permutation(G, xcds):
    assert sorted(logical(b, G, xcds) for b in range(G)) == list(range(G))


def test_owner_is_largest_start_at_or_below():
    for T, G in [(10, 3), (1296, 768), (162, 162), (28224, 1024), (7, 7)]:
        for i in range(T):
            g = owner(i, T, G)
            assert start(g, T, G) <= i < start(g + 1, T, G)
