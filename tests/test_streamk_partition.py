"""The work partition of the contraction kernels, checked on the CPU with
the kernels' own integer maps (paper_1904_05347_amd/csrc/pk_partition.hpp,
built for the host by hipcc into a small shared library).

Stream-K gives logical work-group g the (tile, K-block) iterations
[start(g), start(g+1)); the kernel walks them as segments that end at tile
boundaries, finds a tile's contributors with owner() and stores partial
tiles in slot() (2g for the range's first tile, 2g+1 for its last).  Checked
over many shapes: every iteration is computed exactly once, owner() names
exactly the work-groups that hold a segment of the tile, partial slots never
collide and stay below 2G, and the XCD renumberings of work-group ids (tiles
and stream-K ranges) and the column-strip tile order are permutations.
"""
import ctypes
import itertools
import os
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SHIM_SRC = os.path.join(ROOT, "tests", "partition_shim.cpp")
HEADER = os.path.join(ROOT, "paper_1904_05347_amd", "csrc", "pk_partition.hpp")


@pytest.fixture(scope="module")
def shim(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("shim") / "libpartition_shim.so")
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    subprocess.run([hipcc, "--cuda-host-only", "-x", "hip", "-O1", "-std=c++20", "-shared", "-fPIC",
                    SHIM_SRC, "-o", out], check=True, capture_output=True)
    lib = ctypes.CDLL(out)
    lib.shim_tile_of.argtypes = [ctypes.c_int] * 4 + [ctypes.POINTER(ctypes.c_int)] * 2
    return lib


def start(lib, g, T, G, nkb=1):
    return lib.shim_sk_start(T, G, nkb, g)


def owner(lib, i, T, G, nkb=1):
    return lib.shim_sk_owner(T, G, nkb, i)


def slot(lib, g, t, T, G, nkb):
    return lib.shim_sk_slot(T, G, nkb, g, t)


def segments(lib, g, T, G, nkb):
    """The (tile, kbeg, kend) segments work-group g walks: its range cut at
    tile boundaries, as the kernels walk it."""
    seg, end = start(lib, g, T, G, nkb), start(lib, g + 1, T, G, nkb)
    out = []
    while seg < end:
        tile = seg // nkb
        kbeg = seg - tile * nkb
        kend = min(nkb, kbeg + (end - seg))
        out.append((tile, kbeg, kend))
        seg += kend - kbeg
    return out


CASES = [(tiles, nkb, G) for tiles, nkb, G in itertools.product(
    [1, 2, 3, 7, 52, 196, 785], [1, 2, 5, 18, 72, 144], [1, 8, 24, 256, 512, 768, 1024])
    if G <= tiles * nkb]


@pytest.mark.parametrize("tiles,nkb,G", CASES)
def test_streamk_partition(shim, tiles, nkb, G):
    T = tiles * nkb
    covered = [0] * T
    holders = {}          # tile -> work-groups with a segment in it
    slots = {}
    for g in range(G):
        segs = segments(shim, g, T, G, nkb)
        assert segs, "every work-group has at least one iteration"
        for tile, kbeg, kend in segs:
            assert 0 <= kbeg < kend <= nkb
            for k in range(kbeg, kend):
                covered[tile * nkb + k] += 1
            holders.setdefault(tile, []).append((g, kbeg, kend))
    assert all(c == 1 for c in covered)
    for tile, hs in holders.items():
        lo, hi = owner(shim, tile * nkb, T, G, nkb), owner(shim, tile * nkb + nkb - 1, T, G, nkb)
        assert [g for g, _, _ in hs] == list(range(lo, hi + 1))
        # contributors in increasing g hold increasing K-blocks: the kernel's
        # summation order g = lo .. hi is the order of the reduction
        assert [k for _, k, _ in hs] == sorted(k for _, k, _ in hs)
        full = len(hs) == 1
        assert full == (hs[0][1] == 0 and hs[0][2] == nkb)
        if not full:
            for g, _, _ in hs:
                s = slot(shim, g, tile, T, G, nkb)
                assert 0 <= s < 2 * G
                assert s not in slots, (g, tile, slots.get(s))
                slots[s] = (g, tile)


@pytest.mark.parametrize("G,xcds", [(8, 8), (512, 8), (768, 8), (24, 8), (7, 8), (256, 1)])
def test_xcd_renumbering_is_a_permutation(shim, G, xcds):
    assert sorted(shim.shim_sk_logical(b, G, xcds) for b in range(G)) == list(range(G))


@pytest.mark.parametrize("num,xcds", [(1, 8), (7, 8), (8, 8), (196, 8), (1024, 8), (1025, 8), (52, 1)])
def test_tile_xcd_renumbering_is_a_permutation(shim, num, xcds):
    """Each XCD (work-groups pid % xcds) receives a contiguous run of logical tiles."""
    got = [shim.shim_xcd_tile(pid, num, xcds) for pid in range(num)]
    assert sorted(got) == list(range(num))
    for x in range(min(xcds, num)):
        run = sorted(got[pid] for pid in range(x, num, xcds))
        assert run == list(range(run[0], run[0] + len(run)))


@pytest.mark.parametrize("tiles_m,tiles_n,group_m", [(16, 16, 8), (13, 4, 8), (7, 5, 3), (1, 9, 8), (100, 1, 8)])
def test_tile_order_is_a_permutation(shim, tiles_m, tiles_n, group_m):
    tm, tn = ctypes.c_int(), ctypes.c_int()
    seen = set()
    for t in range(tiles_m * tiles_n):
        shim.shim_tile_of(tiles_m, tiles_n, group_m, t, ctypes.byref(tm), ctypes.byref(tn))
        assert 0 <= tm.value < tiles_m and 0 <= tn.value < tiles_n
        seen.add((tm.value, tn.value))
    assert len(seen) == tiles_m * tiles_n


def test_owner_is_largest_start_at_or_below(shim):
    for T, G in [(10, 3), (1296, 768), (162, 162), (28224, 1024), (7, 7)]:
        for i in range(T):
            g = owner(shim, i, T, G)
            assert start(shim, g, T, G) <= i < start(shim, g + 1, T, G)
