"""GEMM on the GPU through the C-ABI against the CPU oracle."""
import itertools

import numpy as np
import pytest

import oracle
from paper_1904_05347_amd import workloads as wl
from tests.gpu_util import assert_parity, dev, host, require_gpu, sample_rows_cols

pytestmark = pytest.mark.gpu


def _gemm_case(torch, pk, ta, tb, M, N, K, alpha, beta, seed, kind="uniform", slack=0, force=None):
    rng = np.random.default_rng(seed)
    draw = wl.uniform if kind == "uniform" else wl.integers
    a_rows, a_cols = (K, M) if ta == "T" else (M, K)
    b_rows, b_cols = (N, K) if tb == "T" else (K, N)
    A = draw(rng, a_rows * (a_cols + slack)).reshape(a_rows, a_cols + slack)
    B = draw(rng, b_rows * (b_cols + slack)).reshape(b_rows, b_cols + slack)
    C = draw(rng, M * (N + slack)).reshape(M, N + slack)
    dA, dB, dC = dev(A), dev(B), dev(C)
    if force:
        pk.force_config(force)
    try:
        st = pk.binding.sgemm(ta, tb, M, N, K, alpha, dA.data_ptr(), A.shape[1], dB.data_ptr(), B.shape[1],
                              beta, dC.data_ptr(), C.shape[1], torch.cuda.current_stream().cuda_stream)
    finally:
        if force:
            pk.force_config(None)
    assert st == 0, (st, pk.last_invalid_param())
    cfg = pk.last_config_name()
    out = host(dC)
    ref, scale = oracle.sgemm(ta, tb, M, N, K, alpha, A, A.shape[1], B, B.shape[1], beta, C, C.shape[1])
    # the slack columns of C must be untouched
    assert np.array_equal(out[:, N:], C[:, N:])
    return out[:, :N], ref, scale, C[:, :N], cfg


def test_gemm_512_parity():
    torch, pk = require_gpu()
    case = wl.GEMM_SMALL
    A, B, C = case.inputs()
    C = np.full_like(C, np.nan)  # beta == 0: C must not be read
    dA, dB, dC = dev(A), dev(B), dev(C)
    pk.gemm(dA, dB, dC, alpha=1.0, beta=0.0)
    out = host(dC)
    ref, scale = oracle.sgemm("N", "N", 512, 512, 512, 1.0, A, 512, B, 512, 0.0, C, 512)
    mx = assert_parity(out, ref, scale, case.name)
    assert mx < 1e-6


def test_gemm_512_integer_exact():
    torch, pk = require_gpu()
    out, ref, _, _, cfg = _gemm_case(torch, pk, "N", "N", 512, 512, 512, 1.0, 0.0, 101, kind="int")
    assert np.array_equal(out.astype(np.float64), ref), cfg


@pytest.mark.parametrize("ta,tb", list(itertools.product("NT", "NT")))
def test_gemm_transposes_integer_exact(ta, tb):
    torch, pk = require_gpu()
    # several tiles plus ragged tails in M and N; K a multiple of 4 (16-byte path)
    out, ref, _, _, cfg = _gemm_case(torch, pk, ta, tb, 300, 268, 132, 1.0, 0.5, 7, kind="int")
    assert np.array_equal(out.astype(np.float64), ref), (ta, tb, cfg)


EDGE = [1, 3, 17, 63, 65, 129]


@pytest.mark.parametrize("ta,tb", list(itertools.product("NT", "NT")))
def test_gemm_edge_shapes(ta, tb):
    torch, pk = require_gpu()
    rng = np.random.default_rng(hash((ta, tb)) % 1000)
    shapes = [(m, n, k) for m in EDGE for n in EDGE for k in (1, 2, 17, 65)]
    picks = [shapes[i] for i in rng.choice(len(shapes), 24, replace=False)] + [(129, 129, 129), (1, 1, 1)]
    for M, N, K in picks:
        out, ref, scale, C, cfg = _gemm_case(torch, pk, ta, tb, M, N, K, 1.5, -0.5, M * 7 + N * 3 + K, slack=3)
        assert_parity(out, ref, scale, "%s%s %dx%dx%d %s" % (ta, tb, M, N, K, cfg),
                      extra=np.abs(0.5 * C.astype(np.float64)))


def test_gemm_quick_returns():
    torch, pk = require_gpu()
    M, N, K = 70, 33, 20
    rng = np.random.default_rng(5)
    A = wl.uniform(rng, M * K).reshape(M, K)
    B = wl.uniform(rng, K * N).reshape(K, N)
    C = wl.uniform(rng, M * N).reshape(M, N)
    # alpha == 0: C <- beta C, A/B not read (NaN there must not leak)
    dA = dev(np.full_like(A, np.nan))
    dB = dev(np.full_like(B, np.nan))
    dC = dev(C)
    pk.gemm(dA, dB, dC, alpha=0.0, beta=0.5)
    assert np.array_equal(host(dC), (C * np.float32(0.5)))
    # K == 0: C <- beta C
    dC = dev(C)
    st = pk.binding.sgemm("N", "N", M, N, 0, 1.0, None, 1, None, N, 2.0, dC.data_ptr(), N)
    assert st == 0
    assert np.array_equal(host(dC), C * np.float32(2.0))
    # beta == 0 with alpha == 0 writes zeros even over NaN
    dC = dev(np.full_like(C, np.nan))
    pk.gemm(dev(A), dev(B), dC, alpha=0.0, beta=0.0)
    assert np.array_equal(host(dC), np.zeros_like(C))
    # M == 0 / N == 0: nothing happens
    assert pk.binding.sgemm("N", "N", 0, N, K, 1.0, None, K, None, N, 0.0, None, N) == 0
    assert pk.binding.sgemm("N", "N", M, 0, K, 1.0, None, K, None, 1, 0.0, None, 1) == 0


def test_gemm_deterministic_and_streams():
    torch, pk = require_gpu()
    case = wl.GEMM_SWEEP[0]
    A, B, C = case.inputs()
    dA, dB = dev(A), dev(B)
    outs = []
    s = torch.cuda.Stream()
    for stream in (None, s):
        dC = dev(C)
        if stream is None:
            pk.gemm(dA, dB, dC, alpha=1.0, beta=0.5)
        else:
            stream.wait_stream(torch.cuda.current_stream())
            with torch.cuda.stream(stream):
                pk.gemm(dA, dB, dC, alpha=1.0, beta=0.5)
            torch.cuda.current_stream().wait_stream(stream)
        outs.append(host(dC))
    assert np.array_equal(outs[0], outs[1])
    rows, cols = sample_rows_cols(1024, 1024, 2000, 3)
    ref, scale = oracle.sgemm_at("N", "N", 1024, 1024, 1024, 1.0, A, 1024, B, 1024, 0.5, C, 1024, rows, cols)
    assert_parity(outs[0][rows, cols], ref, scale, case.name)


def test_every_gemm_config_forced():
    torch, pk = require_gpu()
    for cfg in pk.configs():
        # stream-K runs through the convolution call only; B-resident forms
        # take only K == bk and N == bn (tested on their own)
        if cfg["kind"] != 0 or cfg["streamk"] or cfg["bres"]:
            continue
        ta = "T" if cfg["trans_a"] else "N"
        tb = "T" if cfg["trans_b"] else "N"
        for M, N, K in [(200, 136, 72), (64, 64, 16), (4, 260, 36)]:
            out, ref, scale, C, used = _gemm_case(torch, pk, ta, tb, M, N, K, 1.0, 0.5, M + N + K,
                                                  kind="int", force=cfg["name"])
            assert used == cfg["name"]
            assert np.array_equal(out.astype(np.float64), ref), (cfg["name"], M, N, K)


def test_gemm_workspace_splits_and_streamk():
    """pk_sgemm_ws: every GEMM configuration that splits K across
    work-groups (tiled, persistent, K-split forms: forced splits of 2 and 3,
    the last slice ragged) and every stream-K form, on integer data with
    beta = 0.5: the slices added in a fixed order must equal the oracle bit
    for bit, twice in a row (a workspace reused with stale contents)."""
    torch, pk = require_gpu()
    ran = 0
    ws = torch.empty(256 << 18, dtype=torch.float32, device="cuda")  # 256 MiB
    for cfg in pk.configs():
        if cfg["kind"] != 0 or cfg["bres"]:
            continue
        ta = "T" if cfg["trans_a"] else "N"
        tb = "T" if cfg["trans_b"] else "N"
        for M, N, K in [(132, 68, 1000), (36, 200, 92)]:
            rng = np.random.default_rng(M * 5 + N + K)
            A = wl.integers(rng, M * K).reshape((K, M) if ta == "T" else (M, K))
            B = wl.integers(rng, K * N).reshape((N, K) if tb == "T" else (K, N))
            C = wl.integers(rng, M * N).reshape(M, N)
            ref, _ = oracle.sgemm(ta, tb, M, N, K, 1.0, A, A.shape[1], B, B.shape[1], 0.5, C, N)
            dA, dB = dev(A), dev(B)
            for splits in ((0,) if cfg["streamk"] else (2, 3)):
                for rep in range(2):
                    dC = dev(C)
                    pk.force_config(cfg["name"])
                    pk.force_splits(splits)
                    try:
                        st = pk.binding.sgemm_ws(ta, tb, M, N, K, 1.0, dA.data_ptr(), A.shape[1], dB.data_ptr(),
                                                 B.shape[1], 0.5, dC.data_ptr(), N, ws.data_ptr(), ws.numel() * 4)
                        used = pk.last_config_name()
                    finally:
                        pk.force_config(None)
                        pk.force_splits(0)
                    if st == 2:  # this configuration does not take these operands
                        break
                    assert st == 0 and used == cfg["name"], (cfg["name"], st)
                    assert np.array_equal(host(dC).astype(np.float64), ref), (cfg["name"], M, N, K, splits, rep)
                    ran += 1
    assert ran >= 400


@pytest.mark.parametrize("cfg,M,N,K,ldc", [
    ("gemm_64x64x16_w2x2_nn_v11", 37, 27, 816, 29),    # 51 K-blocks; rows of 27: one element per work-item
    ("gemm_64x64x32_w2x2_nn_v44", 40, 36, 1088, 44)])  # 34 K-blocks; 16-byte elements, padded rows
def test_split_reduce_widths_and_batches(cfg, M, N, K, ldc):
    """The split-K reduce on both element widths, with splits that fill its
    batches of eight in-flight partials partly (2, 9) and exactly twice
    (17): K is chosen so that each requested split is a whole number of
    K-blocks per slice, and the last requested slice must have been written.
    C's rows are padded: integer data, bit-exact against the oracle, and the
    padding columns untouched."""
    torch, pk = require_gpu()
    rng = np.random.default_rng(M + N + K)
    A = wl.integers(rng, M * K).reshape(M, K)
    B = wl.integers(rng, K * N).reshape(K, N)
    C = np.full((M, ldc), 7.0, dtype=np.float32)
    C[:, :N] = wl.integers(rng, M * N).reshape(M, N)
    ref, _ = oracle.sgemm("N", "N", M, N, K, 1.0, A, K, B, N, 0.5, np.ascontiguousarray(C[:, :N]), N)
    ws = torch.empty(17 * M * N + 64, dtype=torch.float32, device="cuda")
    dA, dB = dev(A), dev(B)
    for splits in (2, 9, 17):
        dC = dev(C)
        ws.fill_(float("nan"))
        pk.force_config(cfg)
        pk.force_splits(splits)
        try:
            st = pk.binding.sgemm_ws("N", "N", M, N, K, 1.0, dA.data_ptr(), K, dB.data_ptr(), N, 0.5,
                                     dC.data_ptr(), ldc, ws.data_ptr(), ws.numel() * 4)
            used = pk.last_config_name()
        finally:
            pk.force_config(None)
            pk.force_splits(0)
        assert st == 0 and used == cfg, (cfg, st, used)
        out = host(dC)
        assert np.array_equal(out[:, :N].astype(np.float64), ref), (cfg, splits)
        assert np.all(out[:, N:] == 7.0), (cfg, splits)
        # slice splits-1 holds partial sums (the split was not rounded down)
        last = host(ws[(splits - 1) * M * N: splits * M * N])
        assert np.all(np.isfinite(last)), (cfg, splits)
        if splits < 17:
            assert np.all(np.isnan(host(ws[splits * M * N: (splits + 1) * M * N]))), (cfg, splits)


@pytest.mark.parametrize("M,N,K", [(64, 64, 1024), (1024, 64, 512), (256, 1024, 1024), (100, 36, 2000)])
def test_gemm_default_workspace(M, N, K):
    """The default choice with the workspace the binding allocates (a split
    across work-groups for these few-tile, long-K products) against the
    oracle on random data."""
    torch, pk = require_gpu()
    need = pk.binding.sgemm_workspace_bytes("N", "N", M, N, K)
    assert need > 0
    rng = np.random.default_rng(M + 3 * N + K)
    A = wl.uniform(rng, M * K).reshape(M, K)
    B = wl.uniform(rng, K * N).reshape(K, N)
    C = wl.uniform(rng, M * N).reshape(M, N)
    dC = dev(C)
    pk.gemm(dev(A), dev(B), dC, alpha=1.5, beta=-0.5)
    ref, scale = oracle.sgemm("N", "N", M, N, K, 1.5, A, K, B, N, -0.5, C, N)
    assert_parity(host(dC), ref, scale, "gemm %dx%dx%d %s" % (M, N, K, pk.last_config_name()))


def test_ksplit_configs():
    """K split among groups of waves inside the work-group: a long reduction
    that does not divide into the groups' K-blocks (groups past the end add
    zeros), ragged tiles, every layout; integer data, so the partial tiles
    added in group order must equal the oracle bit for bit; with beta = 0 and
    C prefilled with NaN every output must be written."""
    torch, pk = require_gpu()
    ran = 0
    for cfg in pk.configs():
        if cfg["kind"] != 0 or cfg["kgroups"] == 1:
            continue
        ta = "T" if cfg["trans_a"] else "N"
        tb = "T" if cfg["trans_b"] else "N"
        # multiples of 4 (the 4-wide loads), ragged against tiles and K-blocks
        for M, N, K, beta in [(132, 68, 1000, 0.5), (64, 64, 1024, 0.0), (36, 200, 92, 0.0)]:
            rng = np.random.default_rng(M * 7 + N + K)
            A = wl.integers(rng, M * K).reshape((K, M) if ta == "T" else (M, K))
            B = wl.integers(rng, K * N).reshape((N, K) if tb == "T" else (K, N))
            C = wl.integers(rng, M * N).reshape(M, N) if beta else np.full((M, N), np.nan, np.float32)
            dA, dB, dC = dev(A), dev(B), dev(C)
            pk.force_config(cfg["name"])
            try:
                st = pk.binding.sgemm(ta, tb, M, N, K, 1.0, dA.data_ptr(), A.shape[1], dB.data_ptr(), B.shape[1],
                                      beta, dC.data_ptr(), N)
                used = pk.last_config_name()
            finally:
                pk.force_config(None)
            assert st == 0 and used == cfg["name"]
            ref, _ = oracle.sgemm(ta, tb, M, N, K, 1.0, A, A.shape[1], B, B.shape[1], beta,
                                  C if beta else np.zeros((M, N), np.float32), N)
            assert np.array_equal(host(dC).astype(np.float64), ref), (cfg["name"], M, N, K)
            ran += 1
    assert ran >= 36


# One shape per branch of the GEMM selection rules, none of them in the
# built-in table, with the configuration each branch picks (the workspace the
# library asks for, so the rules' splits run too).
RULE_SHAPES = [
    ("N", "N", 100, 70, 33, "gemm_64x64x16_w2x2_nn_v11"),              # unaligned: 4-byte loads
    ("T", "T", 300, 260, 96, "gemm_64x64x16_w2x2_tt_v44"),             # TT, few tiles
    ("N", "N", 1000, 128, 64, "gemm_64x64x64_w2x2_nn_v44_br"),         # K = 64: B resident
    ("T", "N", 1000, 128, 64, "gemm_64x64x16_w2x2_tn_v44"),
    ("N", "N", 320, 512, 2048, "gemm_32x64x32_w1x2_k4_nn_v44_dma3"),   # 80 tiles: K split 4 ways inside, 3 across
    ("T", "N", 320, 512, 2048, "gemm_32x64x32_w1x2_k4_tn_v44_d2"),     # (no TN copy form for 32 rows)
    ("N", "T", 320, 512, 2048, "gemm_32x64x32_w1x2_k4_nt_v44_dma3"),
    ("N", "N", 1600, 512, 1024, "gemm_64x64x32_w2x2_k4_nn_v44_dma2"),  # 200 tiles, K >= 1024: four groups
    ("T", "N", 1600, 512, 1024, "gemm_64x64x32_w2x2_k4_tn_v44_dma2"),
    ("N", "T", 1600, 512, 1024, "gemm_64x64x32_w2x2_k4_nt_v44_dma2"),
    ("N", "N", 1600, 512, 512, "gemm_64x64x32_w2x2_k2_nn_v44_dma3"),   # shorter K: two groups
    ("N", "N", 2048, 2048, 128, "gemm_128x128x32_w2x4_nn_v44_o2_dma2"),  # 128 x 128 tiles fill the CUs
    ("N", "N", 20000, 64, 256, "gemm_64x64x32_w2x2_nn_v44_dma2"),      # everything between
    ("T", "N", 20000, 64, 256, "gemm_64x64x32_w2x2_tn_v44_dma2"),
]


@pytest.mark.parametrize("ta,tb,M,N,K,want", RULE_SHAPES,
                         ids=["%s%s_%dx%dx%d" % r[:5] for r in RULE_SHAPES])
def test_gemm_rule_branches(ta, tb, M, N, K, want):
    """Each branch of the selection rules on a shape outside the table: the
    configuration it picks, with its split, equals the oracle bit for bit
    on integer data (beta = 0.5)."""
    torch, pk = require_gpu()
    rng = np.random.default_rng(M + 3 * N + 7 * K)
    A = wl.integers(rng, M * K).reshape((K, M) if ta == "T" else (M, K))
    B = wl.integers(rng, K * N).reshape((N, K) if tb == "T" else (K, N))
    C = wl.integers(rng, M * N).reshape(M, N)
    dC = dev(C)
    pk.gemm(dev(A), dev(B), dC, alpha=1.0, beta=0.5, trans_a=ta == "T", trans_b=tb == "T")
    assert pk.last_config_name() == want
    ref, _ = oracle.sgemm(ta, tb, M, N, K, 1.0, A, A.shape[1], B, B.shape[1], 0.5, C, N)
    assert np.array_equal(host(dC).astype(np.float64), ref), (ta, tb, M, N, K, want)


def test_column_major_swap_identity():
    """A column-major C = A B is the row-major call with operands swapped."""
    torch, pk = require_gpu()
    M, N, K = 96, 80, 40
    rng = np.random.default_rng(9)
    A_cm = wl.integers(rng, M * K).reshape(K, M)  # column-major M x K == row-major K x M buffer
    B_cm = wl.integers(rng, K * N).reshape(N, K)  # column-major K x N
    dA, dB = dev(A_cm), dev(B_cm)
    dC = dev(np.zeros((N, M), np.float32))       # column-major M x N
    st = pk.binding.sgemm("N", "N", N, M, K, 1.0, dB.data_ptr(), K, dA.data_ptr(), M, 0.0, dC.data_ptr(), M)
    assert st == 0
    C_cm = host(dC)
    # the oracle on the same problem stated row-major: A_cm is A^T, B_cm is B^T
    ref, _ = oracle.sgemm("T", "T", M, N, K, 1.0, A_cm, M, B_cm, K, 0.0, np.zeros((M, N), np.float32), N)
    assert np.array_equal(C_cm.T.astype(np.float64), ref)


def test_persistent_configs_loop_over_tiles():
    """Persistent configurations on products with several tiles per resident
    work-group: C starts as NaN with beta = 0, so an unwritten tile shows; the
    sampled outputs (tile corners included) must equal the oracle bit for bit
    on integer data."""
    torch, pk = require_gpu()
    for cfg in pk.configs():
        if cfg["kind"] != 0 or not cfg["persistent"]:
            continue
        ta = "T" if cfg["trans_a"] else "N"
        tb = "T" if cfg["trans_b"] else "N"
        M, N, K = cfg["bm"] * 32, cfg["bn"] * 64 + 4, 44  # ragged last column of tiles
        rng = np.random.default_rng(cfg["bm"] + cfg["bn"])
        A = wl.integers(rng, M * K).reshape((K, M) if ta == "T" else (M, K))
        B = wl.integers(rng, K * N).reshape((N, K) if tb == "T" else (K, N))
        dA, dB = dev(A), dev(B)
        dC = torch.full((M, N), float("nan"), dtype=torch.float32, device="cuda")
        pk.force_config(cfg["name"])
        try:
            pk.gemm(dA, dB, dC, trans_a=ta == "T", trans_b=tb == "T")
            used = pk.last_config_name()
        finally:
            pk.force_config(None)
        assert used == cfg["name"]
        out = host(dC)
        assert np.all(np.isfinite(out)), cfg["name"]
        rows, cols = sample_rows_cols(M, N, 4000, 5, tiles=(cfg["bm"], cfg["bn"]))
        ref, _ = oracle.sgemm_at(ta, tb, M, N, K, 1.0, A, A.shape[1], B, B.shape[1], 0.0,
                                 np.zeros((1, 1), np.float32), N, rows, cols)
        assert np.array_equal(out[rows, cols].astype(np.float64), ref), cfg["name"]


@pytest.mark.parametrize("case", wl.gemm_sweep(), ids=lambda c: c.name)
def test_paper_gemm_sweep(case):
    """The paper's sweep (M, N, K powers of two in [64, 1024]), whole outputs."""
    torch, pk = require_gpu()
    A, B, C = case.inputs()
    dC = dev(np.full_like(C, np.nan))
    pk.gemm(dev(A), dev(B), dC)
    out = host(dC)
    ref, scale = oracle.sgemm("N", "N", case.M, case.N, case.K, 1.0, A, case.lda, B, case.ldb, 0.0, C, case.ldc)
    assert_parity(out, ref, scale, case.name + " " + pk.last_config_name())


def test_streamk_configs_refused_by_sgemm():
    """Stream-K needs a workspace, which pk_sgemm does not take: a forced
    stream-K configuration is refused with PK_ERR_WORKSPACE (as pk_sgemm_ws
    with none)."""
    torch, pk = require_gpu()
    name = next(c["name"] for c in pk.configs() if c["streamk"] and c["kind"] == 0)
    a = torch.ones((64, 64), dtype=torch.float32, device="cuda")
    c = torch.zeros((64, 64), dtype=torch.float32, device="cuda")
    pk.force_config(name)
    try:
        st = pk.binding.sgemm("N", "N", 64, 64, 64, 1.0, a.data_ptr(), 64, a.data_ptr(), 64, 0.0, c.data_ptr(), 64)
    finally:
        pk.force_config(None)
    assert st == 3


def test_bres_configs():
    """B-resident streaming configurations: the 1x1 convolution path and
    pk_sgemm with beta != 0 and leading-dimension slack, on row counts that
    leave a ragged last tile and several tiles per work-group, with N one,
    two and four column blocks; integer data, so every output must equal the
    oracle bit for bit; a product whose K differs from the K-block or whose N
    is not a multiple of the column block is refused."""
    torch, pk = require_gpu()
    ran = 0
    for cfg in pk.configs():
        if not cfg["bres"]:
            continue
        K = cfg["bk"]
        for M, N in ((cfg["bm"] * 3 + 5, cfg["bn"]), (300 * cfg["bm"] + 17, cfg["bn"]),
                     (40 * cfg["bm"] + 9, 2 * cfg["bn"]), (300 * cfg["bm"] + 3, 4 * cfg["bn"])):
            rng = np.random.default_rng(M + N)
            A = wl.integers(rng, M * K).reshape(M, K)
            B = wl.integers(rng, K * N).reshape(K, N)
            # as a 1x1 convolution (image M x 1 x 1 pixels of K channels)
            x = A.reshape(M, 1, 1, K)
            f = B.reshape(1, 1, K, N)
            y = torch.full((M, 1, 1, N), float("nan"), dtype=torch.float32, device="cuda")
            pk.force_config(cfg["name"])
            try:
                pk.conv2d_fwd(dev(x), dev(f), padding="VALID", out=y)
                assert pk.last_config_name() == cfg["name"]
            finally:
                pk.force_config(None)
            ref, _ = oracle.sgemm("N", "N", M, N, K, 1.0, A, K, B, N, 0.0, None, N)
            assert np.array_equal(host(y).reshape(M, N).astype(np.float64), ref), cfg["name"]
            ran += 1
        # pk_sgemm, beta = 0.5, lda / ldb / ldc with slack (the slack of C untouched)
        M, N = 5 * cfg["bm"] + 3, 2 * cfg["bn"]
        rng = np.random.default_rng(7 * N)
        A = wl.integers(rng, M * (K + 8)).reshape(M, K + 8)
        B = wl.integers(rng, K * (N + 4)).reshape(K, N + 4)
        C = wl.integers(rng, M * (N + 12)).reshape(M, N + 12)
        dA, dB, dC = dev(A), dev(B), dev(C)  # held: a freed temporary's memory is handed out again
        pk.force_config(cfg["name"])
        try:
            st = pk.binding.sgemm("N", "N", M, N, K, 1.0, dA.data_ptr(), K + 8, dB.data_ptr(), N + 4, 0.5,
                                  dC.data_ptr(), N + 12)
            torch.cuda.synchronize()
            st_bad = pk.binding.sgemm("N", "N", M, N, K // 2, 1.0, dA.data_ptr(), K + 8, dB.data_ptr(),
                                      N + 4, 0.5, dC.data_ptr(), N + 12)
            st_bad_n = pk.binding.sgemm("N", "N", M, N - 4, K, 1.0, dA.data_ptr(), K + 8, dB.data_ptr(),
                                        N + 4, 0.5, dC.data_ptr(), N + 12)
        finally:
            pk.force_config(None)
        assert st == 0 and st_bad == 2 and st_bad_n == 2
        out = host(dC)
        ref, _ = oracle.sgemm("N", "N", M, N, K, 1.0, A, K + 8, B, N + 4, 0.5, C, N + 12)
        assert np.array_equal(out[:, :N].astype(np.float64), ref), cfg["name"]
        assert np.array_equal(out[:, N:], C[:, N:]), cfg["name"]
    assert ran >= 16
