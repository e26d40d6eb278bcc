"""The C-ABI library on the CPU: it loads, exports every declared symbol, and
its host-side logic (argument checks, output sizes, padding, the compiled
tile-parameter space) behaves as documented.  No call here reaches the GPU:
every call either is host-only or fails validation before any launch."""
import ctypes
import os
import re

import pytest

import oracle
from tests import pins

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pk.h")


@pytest.fixture(scope="module")
def pk():
    import paper_1904_05347_amd as pk
    from paper_1904_05347_amd import binding
    if not os.path.exists(binding.LIB_PATH):
        from paper_1904_05347_amd import build
        build.build(verbose=False)
    pk.load()
    return pk


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pk_[a-z0-9_]+)\s*\(", text)))


def test_header_symbols_exported(pk):
    from paper_1904_05347_amd import binding
    names = declared_functions()
    assert len(names) >= 10
    lib = ctypes.CDLL(binding.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(binding.SIGNATURES), "binding and header disagree"


def test_out_dims_and_same_pads_match_oracle_and_tables(pk):
    for name in ("vgg16_layers.csv", "resnet50_layers.csv"):
        for row in pins.read_golden(name):
            k, s = int(row["window"]), int(row["stride"])
            H, W = int(row["in_h"]), int(row["in_w"])
            pads = (0, 0, 0, 0) if k == 7 else pk.conv2d_same_pads(H, W, k, k, s, s)
            assert pads == ((0, 0, 0, 0) if k == 7 else oracle.same_pads(H, W, k, k, s, s))
            assert pk.conv2d_out_dims(H, W, k, k, s, s, *pads) == (int(row["out_h"]), int(row["out_w"]))
    for H in range(1, 10):
        for k in range(1, 6):
            for s in range(1, 4):
                assert pk.conv2d_same_pads(H, H + 2, k, k, s, s) == oracle.same_pads(H, H + 2, k, k, s, s)
                for pads in [(0, 0, 0, 0), (1, 2, 0, 1), (2, 2, 2, 2)]:
                    try:
                        want = oracle.conv2d_out_dims(H, H + 2, k, k, s, s, *pads)
                    except ValueError:
                        with pytest.raises(pk.PkError):
                            pk.conv2d_out_dims(H, H + 2, k, k, s, s, *pads)
                        continue
                    assert pk.conv2d_out_dims(H, H + 2, k, k, s, s, *pads) == want


def _gemm_status(pk, *args):
    from paper_1904_05347_amd import binding
    st = binding.sgemm(*args)
    return st, pk.last_invalid_param()


def test_gemm_argument_checks(pk):
    fake = 0x10000  # never dereferenced: every call below fails validation or is empty
    ok = ("N", "N", 4, 5, 6, 1.0, fake, 6, fake + 4096, 5, 0.0, fake + 8192, 5)
    cases = [
        ((b"X",) + ok[1:], 1),
        (ok[:1] + (b"Q",) + ok[2:], 2),
        (ok[:2] + (-1,) + ok[3:], 3),
        (ok[:3] + (-1,) + ok[4:], 4),
        (ok[:4] + (-1,) + ok[5:], 5),
        (ok[:7] + (5,) + ok[8:], 8),     # lda < K
        (ok[:9] + (4,) + ok[10:], 10),   # ldb < N
        (ok[:12] + (4,), 13),            # ldc < N
        (("T",) + ok[1:7] + (3,) + ok[8:], 8),   # 'T': lda < M
        (ok[:1] + ("T",) + ok[2:9] + (5,) + ok[10:], 10),  # 'T': ldb < K
        (ok[:11] + (None,) + ok[12:], 12),       # C missing
        (ok[:6] + (None,) + ok[7:], 7),          # A missing
        (ok[:8] + (None,) + ok[9:], 9),          # B missing
        (ok[:11] + (fake + 16,) + ok[12:], 12),  # C overlaps A
    ]
    for args, pos in cases:
        st, p = _gemm_status(pk, *args)
        assert (st, p) == (1, pos), (args, st, p)
    # empty problems return before touching anything
    assert _gemm_status(pk, "N", "N", 0, 5, 6, 1.0, None, 6, None, 5, 0.0, None, 5)[0] == 0
    assert _gemm_status(pk, "n", "c", 4, 0, 6, 1.0, None, 6, None, 6, 0.0, None, 1)[0] == 0


def test_conv_argument_checks(pk):
    from paper_1904_05347_amd import binding
    fake = 0x10000
    good = dict(x=fake, N=1, H=5, W=5, Cin=4, f=fake + (1 << 20), KH=3, KW=3, Cout=4, sh=1, sw=1,
                pt=1, pl=1, pb=1, pr=1, y=fake + (2 << 20), Ho=5, Wo=5)
    order = list(good)
    bad = [("N", -1, 2), ("H", 0, 3), ("W", 0, 4), ("Cin", 0, 5), ("KH", 0, 7), ("KW", 0, 8),
           ("Cout", 0, 9), ("sh", 0, 10), ("sw", 0, 11), ("pt", -1, 12), ("pl", -1, 13),
           ("pb", -1, 14), ("pr", -1, 15), ("Ho", 4, 17), ("Wo", 6, 18), ("KH", 9, 7), ("KW", 8, 8),
           ("x", None, 1), ("f", None, 6), ("y", None, 16), ("y", fake + 64, 16)]
    for key, val, pos in bad:
        args = dict(good)
        args[key] = val
        st = binding.conv2d_fwd_raw(*[args[k] for k in order])
        assert (st, pk.last_invalid_param()) == (1, pos), (key, val, st, pk.last_invalid_param())
    args = dict(good, N=0)
    assert binding.conv2d_fwd_raw(*[args[k] for k in order]) == 0


def test_winograd_argument_checks(pk):
    """Host-side checks of pk_conv2d_winograd_fwd: the positions of
    pk_conv2d_fwd, then the window / stride it supports and its workspace."""
    from paper_1904_05347_amd import binding
    fake = 0x10000
    N, H, W, Cin, Cout = 2, 5, 7, 6, 10
    need = pk.conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, 1, 1, 1, 1)
    # U (16 Cin Cout), V (16 T Cin), M (16 T Cout) floats, T = N ceil(Ho/2) ceil(Wo/2)
    T = N * 3 * 4
    floor = 4 * 16 * (Cin * Cout + T * Cin + T * Cout)
    assert floor <= need < floor + 3 * 256, (need, floor)
    ws = fake + (8 << 20)
    good = dict(x=fake, N=N, H=H, W=W, Cin=Cin, f=fake + (1 << 20), KH=3, KW=3, Cout=Cout, sh=1, sw=1,
                pt=1, pl=1, pb=1, pr=1, y=fake + (2 << 20), Ho=5, Wo=7, ws=ws, ws_bytes=need)
    order = list(good)

    def call(**kw):
        args = dict(good, **kw)
        return binding.conv2d_winograd_raw(*[args[k] for k in order])

    bad = [("N", -1, 2), ("H", 0, 3), ("W", 0, 4), ("Cin", 0, 5), ("KH", 0, 7), ("KW", 0, 8),
           ("Cout", 0, 9), ("sh", 0, 10), ("sw", 0, 11), ("pt", -1, 12), ("pl", -1, 13),
           ("pb", -1, 14), ("pr", -1, 15), ("Ho", 4, 17), ("Wo", 6, 18),
           ("x", None, 1), ("f", None, 6), ("y", None, 16), ("y", fake + 64, 16)]
    for key, val, pos in bad:
        st = call(**{key: val})
        assert (st, pk.last_invalid_param()) == (1, pos), (key, val, st, pk.last_invalid_param())
    # windows and strides other than 3 x 3, stride 1
    assert call(KH=5, KW=5, pt=2, pl=2, pb=2, pr=2) == 2
    assert call(KH=1, KW=1, pt=0, pl=0, pb=0, pr=0) == 2
    assert call(sh=2, sw=2, Ho=3, Wo=4) == 2
    # the workspace is required, large enough, aligned and disjoint from the tensors
    assert call(ws=None) == 3
    assert call(ws_bytes=need - 1) == 3
    assert (call(ws=ws + 4), pk.last_invalid_param()) == (1, 19)
    assert (call(ws=fake + (1 << 20) - 64), pk.last_invalid_param()) == (1, 19)
    assert call(N=0) == 0


def test_noalloc_argument_checks(pk):
    """pk_conv2d_fwd_noalloc: the argument positions of pk_conv2d_fwd (all
    checked before the scratch buffer is looked up), and a call whose
    workspace would exceed the static buffer refused before any work."""
    from paper_1904_05347_amd import binding
    fake = 0x10000
    good = dict(x=fake, N=1, H=5, W=5, Cin=4, f=fake + (1 << 20), KH=3, KW=3, Cout=4, sh=1, sw=1,
                pt=1, pl=1, pb=1, pr=1, y=fake + (2 << 20), Ho=5, Wo=5)
    order = list(good)
    bad = [("N", -1, 2), ("H", 0, 3), ("W", 0, 4), ("Cin", 0, 5), ("KH", 0, 7), ("KW", 0, 8),
           ("Cout", 0, 9), ("sh", 0, 10), ("sw", 0, 11), ("pt", -1, 12), ("pl", -1, 13),
           ("pb", -1, 14), ("pr", -1, 15), ("Ho", 4, 17), ("Wo", 6, 18),
           ("x", None, 1), ("f", None, 6), ("y", None, 16), ("y", fake + 64, 16)]
    for key, val, pos in bad:
        args = dict(good)
        args[key] = val
        st = binding.conv2d_fwd_noalloc_raw(*[args[k] for k in order])
        assert (st, pk.last_invalid_param()) == (1, pos), (key, val, st, pk.last_invalid_param())
    assert binding.conv2d_fwd_noalloc_raw(*[dict(good, N=0)[k] for k in order]) == 0
    # a forced split of 2 over 32000 x 512 outputs: 2 x 32000 x 512 partial
    # sums (125 MiB), more than the static buffer (the default choices of
    # this library stay below it: its largest, a stream-K plan, is 64 MiB)
    big = dict(good, H=160, W=200, Cin=64, Cout=512, Ho=160, Wo=200,
               f=fake + (64 << 20), y=fake + (128 << 20))
    pk.force_splits(2)
    try:
        need = pk.conv2d_workspace_bytes(1, 160, 200, 64, 3, 3, 512, 1, 1, 1, 1, 1, 1)
        assert need > binding.NOALLOC_SCRATCH_BYTES, need
        assert binding.conv2d_fwd_noalloc_raw(*[big[k] for k in order]) == binding.PK_ERR_SCRATCH_LIMIT
    finally:
        pk.force_splits(0)
    assert "scratch" in binding.load().pk_status_string(binding.PK_ERR_SCRATCH_LIMIT).decode().lower()
    # the binding's figure is the header's
    header = open(os.path.join(ROOT, "include", "pk.h")).read()
    m = re.search(r"#define PK_NOALLOC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", header)
    assert m and int(m.group(1)) << int(m.group(2)) == binding.NOALLOC_SCRATCH_BYTES
    m = re.search(r"PK_ERR_SCRATCH_LIMIT = (\d+)", header)
    assert m and int(m.group(1)) == binding.PK_ERR_SCRATCH_LIMIT


def test_winograd_tile_argument_checks(pk):
    """pk_conv2d_winograd_tile_fwd: the tile size m at position 19 (2 or 4),
    the workspace at 20, its size from the tile workspace query (36 batched
    matrices of T = N ceil(Ho/4) ceil(Wo/4) rows for m = 4), and the checks of
    pk_conv2d_winograd_fwd before them."""
    from paper_1904_05347_amd import binding
    fake = 0x10000
    N, H, W, Cin, Cout = 2, 5, 7, 6, 10
    need4 = binding.conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, 1, 1, 1, 1, tile=4)
    T4 = N * 2 * 2
    floor4 = 4 * 36 * (Cin * Cout + T4 * Cin + T4 * Cout)
    assert floor4 <= need4 < floor4 + 3 * 256, (need4, floor4)
    assert binding.conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, 1, 1, 1, 1, tile=2) == \
        pk.conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, 1, 1, 1, 1)
    for m in (0, 1, 3, 5, 6):
        assert binding.conv2d_winograd_workspace_bytes(N, H, W, Cin, Cout, 1, 1, 1, 1, tile=m) == 0
    ws = fake + (8 << 20)
    good = dict(x=fake, N=N, H=H, W=W, Cin=Cin, f=fake + (1 << 20), KH=3, KW=3, Cout=Cout, sh=1, sw=1,
                pt=1, pl=1, pb=1, pr=1, y=fake + (2 << 20), Ho=5, Wo=7, m=4, ws=ws, ws_bytes=need4)
    order = list(good)

    def call(**kw):
        args = dict(good, **kw)
        return binding.conv2d_winograd_tile_raw(*[args[k] for k in order])

    bad = [("N", -1, 2), ("Cin", 0, 5), ("KH", 0, 7), ("pt", -1, 12), ("Ho", 4, 17), ("Wo", 6, 18),
           ("x", None, 1), ("f", None, 6), ("y", None, 16), ("m", 3, 19), ("m", 0, 19), ("m", 8, 19)]
    for key, val, pos in bad:
        st = call(**{key: val})
        assert (st, pk.last_invalid_param()) == (1, pos), (key, val, st, pk.last_invalid_param())
    assert call(KH=5, KW=5, pt=2, pl=2, pb=2, pr=2) == 2
    assert call(sh=2, sw=2, Ho=3, Wo=4) == 2
    assert call(ws=None) == 3
    assert call(ws_bytes=need4 - 1) == 3
    assert (call(ws=ws + 4), pk.last_invalid_param()) == (1, 20)
    assert call(N=0) == 0


def test_direct_to_lds_range_checks(pk):
    """The direct-to-LDS forms address one tile's rows of each operand (and
    a convolution's whole image) in 32-bit byte offsets: a forced one is
    refused (PK_ERR_NOT_SUPPORTED) when those rows span 2 GiB or more, and
    accepted up to the launch below that; every call fails before a kernel
    launches (no GPU here), so the refusal is the range check's."""
    from paper_1904_05347_amd import binding
    fake = 0x100000
    big_lda = (1 << 31) // (4 * 256) + 4  # 256 rows of A span just over 2 GiB
    pk.force_config("gemm_256x256x32_w2x4_nn_v44_o2_dma2")
    try:
        st = binding.sgemm("N", "N", 256, 256, 64, 1.0, fake, big_lda, fake + (1 << 40), 256, 0.0,
                           fake + (2 << 40), 256)
        assert st == 2
        # transposed A: BK rows of lda floats per tile, far below the limit
        pk.force_config("gemm_256x256x32_w2x4_tn_v44_o2_dma2")
        st = binding.sgemm("T", "N", 256, 256, 64, 1.0, fake, big_lda, fake + (1 << 40), 256, 0.0,
                           fake + (2 << 40), 256)
        assert st != 2
    finally:
        pk.force_config(None)
    # convolution: an image of 2 GiB or more
    pk.force_config("conv_128x128x32_w2x4_v44_o2_dma2")
    try:
        N, H, W, Cin, Cout = 64, 128, 128, 512, 128  # 4 * N*H*W*Cin = 2 GiB
        st = binding.conv2d_fwd_raw(fake, N, H, W, Cin, fake + (1 << 42), 3, 3, Cout, 1, 1, 1, 1, 1, 1,
                                    fake + (2 << 42), H, W)
        assert st == 2
    finally:
        pk.force_config(None)


def test_gemm_workspace_checks(pk):
    """pk_sgemm_ws: a forced split needs workspace for every slice
    (PK_ERR_WORKSPACE), the workspace must not overlap A, B or C (position 14),
    a B-resident form takes no split; the size query follows the forced
    choice and the rules.  Every call fails before a kernel launches."""
    from paper_1904_05347_amd import binding
    fake = 0x100000
    M, N, K = 64, 64, 1024
    A, B, C = fake, fake + (1 << 22), fake + (2 << 22)
    ws = fake + (4 << 22)
    per_split = M * N * 4

    def call(ws_ptr, ws_bytes):
        st = binding.sgemm_ws("N", "N", M, N, K, 1.0, A, K, B, N, 0.0, C, N, ws_ptr, ws_bytes)
        return st, pk.last_invalid_param()

    pk.force_config("gemm_64x64x32_w2x2_nn_v44")
    pk.force_splits(4)
    try:
        assert binding.sgemm_workspace_bytes("N", "N", M, N, K) == 4 * per_split
        assert call(None, 0)[0] == 3
        assert call(ws, 4 * per_split - 4)[0] == 3
        assert call(A + 64, 4 * per_split) == (1, 14)
        assert call(C - 4 * per_split + 4, 4 * per_split) == (1, 14)
    finally:
        pk.force_config(None)
        pk.force_splits(0)
    pk.force_config("gemm_64x64x64_w2x2_nn_v44_br")
    pk.force_splits(2)
    try:
        st = binding.sgemm_ws("N", "N", M, N, 64, 1.0, A, 64, B, N, 0.0, C, N, ws, 2 * per_split)
        assert st == 2
    finally:
        pk.force_config(None)
        pk.force_splits(0)
    # the rules: a product whose tiles fill the CUs takes no split; a small
    # one with a long K takes one (K-split form, at least two steps per group)
    assert binding.sgemm_workspace_bytes("N", "N", 4096, 4096, 4096) == 0
    assert binding.sgemm_workspace_bytes("N", "N", 64, 64, 64) == 0
    need = binding.sgemm_workspace_bytes("N", "N", 64, 64, 1024)
    assert need > 0 and need % per_split == 0
    # a K-split form (one work-group per CU) never splits past one round of
    # work-groups (256 CUs): 200 tiles of 64 x 64 with K = 2048 take no
    # split, 80 tiles of 32 x 64 a split of 3 (rounding up would take 4)
    assert binding.sgemm_workspace_bytes("N", "N", 1600, 512, 2048) == 0
    assert binding.sgemm_workspace_bytes("N", "N", 320, 512, 2048) == 3 * 320 * 512 * 4


def test_tune_argument_checks(pk):
    """The tuner's own arguments are checked before anything runs."""
    from paper_1904_05347_amd import binding
    lib = pk.load()
    fake = 0x10000
    r = binding.TuneResult()
    st = lib.pk_tune_sgemm(b"N", b"N", 8, 8, 8, 1.0, fake, 8, fake + 4096, 8, 0.0, fake + 8192, 8, None, 0, 0,
                           None, ctypes.byref(r))
    assert (st, pk.last_invalid_param()) == (1, 16)
    st = lib.pk_tune_sgemm(b"N", b"N", 8, 8, 8, 1.0, fake, 8, fake + 4096, 8, 0.0, fake + 8192, 8, None, 0, 3,
                           None, None)
    assert (st, pk.last_invalid_param()) == (1, 18)
    conv = [fake, 1, 5, 5, 4, fake + (1 << 20), 3, 3, 4, 1, 1, 1, 1, 1, 1, fake + (2 << 20), 5, 5, None, 0]
    st = lib.pk_tune_conv2d_fwd(*conv, 0, None, ctypes.byref(r))
    assert (st, pk.last_invalid_param()) == (1, 21)
    st = lib.pk_tune_conv2d_fwd(*conv, 2, None, None)
    assert (st, pk.last_invalid_param()) == (1, 23)
    assert lib.pk_tune_reset() == 0


def test_config_space(pk):
    cfgs = pk.configs()
    assert len(cfgs) >= 10
    names = [c["name"] for c in cfgs]
    assert len(set(names)) == len(names)
    for c in cfgs:
        assert c["threads"] == 64 * c["waves_m"] * c["waves_n"] * c["kgroups"]
        assert c["kgroups"] == 1 or (c["kind"] in (0, 1) and not c["persistent"] and not c["streamk"])
        assert c["lds_bytes"] <= 160 * 1024
        if c["kind"] == 2:  # tiled direct convolution: one LDS input patch
            continue
        assert c["bm"] % (32 * c["waves_m"]) == 0 and c["bn"] % (32 * c["waves_n"]) == 0
        assert c["bk"] % 8 == 0
        if c["dma"]:  # unpadded, swizzled tiles copied straight into 2 to 4 LDS stages
            assert c["kind"] in (0, 1) and c["stages"] in (2, 3, 4) and c["vec_a"] == c["vec_b"] == 4
            assert c["lds_bytes"] == c["kgroups"] * c["stages"] * 4 * (c["bm"] * c["bk"] + c["bk"] * c["bn"]), c["name"]
            assert c["name"].endswith("_dma%d" % c["stages"]) or c["name"].endswith("_dma%d_sk" % c["stages"])
            continue
        assert c["stages"] in (1, 2)
        assert c["stages"] == 2 or (c["kind"] == 0 and c["name"].endswith("_s1"))
        # one or two LDS stages of the A and B tiles, each row padded by 4 floats
        a_k = c["kind"] == 1 or not c["trans_a"]
        a_tile = c["bm"] * (c["bk"] + 4) if a_k else c["bk"] * (c["bm"] + 4)
        b_tile = c["bn"] * (c["bk"] + 4) if c["trans_b"] else c["bk"] * (c["bn"] + 4)
        if c["bres"]:  # two stages of A, and B held whole (n-major)
            assert c["lds_bytes"] == 4 * (2 * a_tile + c["bn"] * (c["bk"] + 4)), c["name"]
            continue
        # K split inside the work-group: every group of waves has its own stages
        assert c["kgroups"] >= 1
        assert c["threads"] == 64 * c["waves_m"] * c["waves_n"] * c["kgroups"] <= 1024, c["name"]
        assert c["lds_bytes"] == c["kgroups"] * c["stages"] * 4 * (a_tile + b_tile), c["name"]
        assert c["lds_bytes"] <= 160 * 1024
    # every GEMM layout has a 16-byte and a scalar-load instance
    for ta in (0, 1):
        for tb in (0, 1):
            vecs = {c["vec_a"] for c in cfgs if c["kind"] == 0 and c["trans_a"] == ta and c["trans_b"] == tb}
            assert {1, 4} <= vecs


def test_selection_names_exist(pk):
    """Every configuration the built-in table or the selection rules name is
    compiled (a misspelt name would silently fall back to the rules): the
    table entries, the convolution rules, and the GEMM rules' name patterns
    for each layout they serve (tiled and direct-to-LDS forms for NN, TN and
    NT, the B-resident form for NN, the scalar-load and TT forms for TT)."""
    names = {c["name"] for c in pk.configs()}
    src = open(os.path.join(ROOT, "paper_1904_05347_amd", "csrc", "pk_api.hip")).read()
    a = src.index("const TunedShape kTuned[] = {")
    table = re.findall(r'"((?:gemm|conv|direct)_[a-z0-9_]+)"', src[a:src.index("};", a)])
    assert len(table) >= 100
    assert set(table) <= names, sorted(set(table) - names)
    conv = src[src.index("const Config *select_conv"):]
    conv = re.findall(r'"(conv_[a-z0-9_]+)"', conv[:conv.index("\n}\n")])
    assert len(conv) >= 5 and set(conv) <= names, sorted(set(conv) - names)
    body = src[src.index("const Config *select_gemm"):]
    body = body[:body.index("\n}\n")]
    # pick(direct-to-LDS form, register-staged twin): the first for NN, and
    # for every layout one of the two (32-row tiles have no TN copy form)
    pairs = re.findall(r'pick\("(gemm_[a-z0-9_%]+)", "(gemm_[a-z0-9_%]+)"\)', body)
    assert len(pairs) >= 5
    for dma, reg in pairs:
        assert dma % "nn" in names, dma % "nn"
        for lay in ("nn", "tn", "nt"):
            assert dma % lay in names or reg % lay in names, (dma % lay, reg % lay)
    single = set(re.findall(r'"(gemm_[a-z0-9_]+%s[a-z0-9_]*)"', body)) - {n for pr in pairs for n in pr}
    assert len(single) >= 4
    for pat in single:
        layouts = ["nn"] if pat.endswith("_br") else ["nn", "tn", "nt", "tt"]
        for lay in layouts:
            assert pat % lay in names, pat % lay


def test_force_config_and_status_strings(pk):
    from paper_1904_05347_amd import binding
    with pytest.raises(pk.PkError):
        pk.force_config("no_such_config")
    pk.force_config(pk.configs()[0]["name"])
    pk.force_config(None)
    with pytest.raises(pk.PkError):
        pk.force_splits(-1)
    lib = binding.load()
    for s in range(5):
        assert lib.pk_status_string(s)
    assert pk.conv2d_workspace_bytes(32, 7, 7, 2048, 3, 3, 512, 1, 1, 1, 1, 1, 1) >= 0


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    """Without libpk.so the package raises instead of computing anything:
    there is no other compute path to fall back to."""
    import paper_1904_05347_amd as pkg
    from paper_1904_05347_amd import binding
    monkeypatch.setattr(binding, "LIB_PATH", str(tmp_path / "libpk.so"))
    monkeypatch.setattr(binding, "_lib", None)
    with pytest.raises(pkg.PkLibraryMissing):
        pkg.load()
    with pytest.raises(pkg.PkLibraryMissing):
        pkg.conv2d_out_dims(8, 8, 3, 3, 1, 1, 1, 1, 1, 1)
